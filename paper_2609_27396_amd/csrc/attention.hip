// Multi-boundary attention of the all-boundary backbone (tree mask of Section 3.2).
//
// Every block row (spine or mask) of a request sees the whole cached context, so the
// context part is plain dense attention shared by all (gamma+1)^2 rows and all query
// heads of a KV group.  It runs as an MFMA flash-attention pass over context chunks:
// one workgroup per (request, KV head, 64 query rows, context chunk) stages the chunk's
// K (keys x head_dim) and V^T (head_dim x keys, the cache stores V transposed) in LDS
// and computes S^T = K Q^T and O^T += V^T P^T with v_mfma_f32_16x16x32_bf16, keeping an
// online softmax in log2 units.  P enters the PV product as a bf16 hi + lo pair (two
// MFMAs), so the probabilities keep ~16 significant bits: a single bf16 rounding of P
// moves the result by about one bf16 ulp of the hidden state, which is as large as the
// whole error budget.  Each chunk emits an unnormalised partial (O, m, l).
//
// The merge kernel (one wave per row and query head) folds the context partials and
// then walks the row's in-block keys under the tree mask -- spine t_j sees t_0..t_j,
// branch r's masks see t_0..t_r and the branch's own masks -- and writes O.
#include <math.h>

#include "common.h"
#include "internal.h"

namespace dpara {
namespace {

constexpr float kLog2e = 1.4426950408889634f;

template <int HD>
__global__ __launch_bounds__(256) void attn_ctx_mfma(AttnArgs a) {
  constexpr int KB = 64;          // keys per staged block
  constexpr int LDKS = HD + 8;    // K tile row stride (bf16)
  constexpr int LDV = KB + 8;     // V^T tile row stride (bf16)
  constexpr int NKS = HD / 32;    // k-steps over head_dim for S
  constexpr int NHB = HD / 16;    // 16-row blocks of head_dim for O^T
  __shared__ __attribute__((aligned(16))) bf16_t Ks[KB * LDKS];
  __shared__ __attribute__((aligned(16))) bf16_t Vs[HD * LDV];

  const int b = blockIdx.z / a.n_kv, kvh = blockIdx.z % a.n_kv;
  const int grp = a.n_q / a.n_kv;
  const int nrows = grp * a.R;
  const int L = min(max(a.ctx_len[b], 0), a.cap);
  const int k_begin = blockIdx.y * a.chunk;
  if (k_begin >= L) return;
  const int k_end = min(L, k_begin + a.chunk);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int lq = lane & 15, g4 = lane >> 4;
  const int qi = blockIdx.x * 64 + wave * 16 + lq;

  // Q^T fragments (B operand): Q[qi][ks*32 + g4*8 + 0..7]
  const bf16_t* Qp = (const bf16_t*)a.Q + (int64_t)(b * a.n_kv + kvh) * nrows * HD;
  bf16x8_t qf[NKS];
#pragma unroll
  for (int ks = 0; ks < NKS; ++ks) {
    if (qi < nrows) qf[ks] = *(const bf16x8_t*)(Qp + (int64_t)qi * HD + ks * 32 + g4 * 8);
    else qf[ks] = bf16x8_t{0, 0, 0, 0, 0, 0, 0, 0};
  }

  f32x4_t o[NHB];
#pragma unroll
  for (int hb = 0; hb < NHB; ++hb) o[hb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY, l_run = 0.f;
  const float sc = kLog2e / sqrtf((float)HD);

  const int64_t kvbase = (int64_t)(b * a.n_kv + kvh);
  const bf16_t* Kg = (const bf16_t*)a.Kc + kvbase * a.cap * HD;
  const bf16_t* Vg = (const bf16_t*)a.Vc + kvbase * HD * a.cap;

  for (int kb0 = k_begin; kb0 < k_end; kb0 += KB) {
    __syncthreads();
    for (int c = threadIdx.x; c < KB * HD / 8; c += 256) {
      const int kr = c / (HD / 8), kc = (c % (HD / 8)) * 8;
      const int key = kb0 + kr;
      uint4 v = make_uint4(0, 0, 0, 0);
      if (key < k_end) v = *(const uint4*)(Kg + (int64_t)key * HD + kc);
      *(uint4*)&Ks[kr * LDKS + kc] = v;
    }
    for (int c = threadIdx.x; c < HD * KB / 8; c += 256) {
      const int d = c / (KB / 8), kc = (c % (KB / 8)) * 8;
      const int key = kb0 + kc;
      const bf16_t* src = Vg + (int64_t)d * a.cap + key;
      uint4 v;
      if (key + 8 <= k_end) {
        v = *(const uint4*)src;
      } else {
        bf16_t t[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) t[j] = (key + j < k_end) ? src[j] : (bf16_t)0;
        v = make_uint4(t[0] | ((uint32_t)t[1] << 16), t[2] | ((uint32_t)t[3] << 16),
                       t[4] | ((uint32_t)t[5] << 16), t[6] | ((uint32_t)t[7] << 16));
      }
      *(uint4*)&Vs[d * LDV + kc] = v;
    }
    __syncthreads();

    // S^T block: s[kb][r] = score(key = kb0 + kb*16 + g4*4 + r, query qi)
    f32x4_t s[4];
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      s[kb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks) {
        const bf16x8_t kf = *(const bf16x8_t*)&Ks[(kb * 16 + lq) * LDKS + ks * 32 + g4 * 8];
        s[kb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qf[ks], s[kb], 0, 0, 0);
      }
    }
    float mx = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int key = kb0 + kb * 16 + g4 * 4 + r;
        const float v = key < k_end ? s[kb][r] * sc : -INFINITY;
        s[kb][r] = v;
        mx = fmaxf(mx, v);
      }
    mx = fmaxf(mx, __shfl_xor(mx, 16, kWave));
    mx = fmaxf(mx, __shfl_xor(mx, 32, kWave));
    const float m_new = fmaxf(m_run, mx);  // finite: key kb0 < k_end is in this block
    const float alpha = exp2f(m_run - m_new);
    float psum = 0.f;
    bf16_t pb[4][4], pl[4][4];  // p = hi + lo, both bf16 (16 significant bits of p)
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float p = exp2f(s[kb][r] - m_new);
        psum += p;
        pb[kb][r] = f2bf(p);
        pl[kb][r] = f2bf(p - bf2f(pb[kb][r]));
      }
    l_run = l_run * alpha + psum;
    m_run = m_new;
#pragma unroll
    for (int hb = 0; hb < NHB; ++hb) o[hb] *= alpha;

    // O^T += V^T P^T over 64 keys = 2 k-steps of 32.  Lane (g4) slot j of k-step t holds
    // key t*32 + g4*4 + j (j < 4) or t*32 + 16 + g4*4 + (j-4): the same key set is used
    // for the V^T operand, so the contraction pairs matching keys.
    // P enters as hi + lo so the product keeps ~16 bits of p (V is exact in bf16).
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      bf16x8_t pf, pfl;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        pf[j] = __builtin_bit_cast(__bf16, pb[2 * t][j]);
        pf[j + 4] = __builtin_bit_cast(__bf16, pb[2 * t + 1][j]);
        pfl[j] = __builtin_bit_cast(__bf16, pl[2 * t][j]);
        pfl[j + 4] = __builtin_bit_cast(__bf16, pl[2 * t + 1][j]);
      }
#pragma unroll
      for (int hb = 0; hb < NHB; ++hb) {
        const bf16_t* vr = &Vs[(hb * 16 + lq) * LDV + t * 32 + g4 * 4];
        const uint2 lo = *(const uint2*)vr;
        const uint2 hi = *(const uint2*)(vr + 16);
        const uint4 packed = make_uint4(lo.x, lo.y, hi.x, hi.y);
        const bf16x8_t vf = __builtin_bit_cast(bf16x8_t, packed);
        o[hb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pf, o[hb], 0, 0, 0);
        o[hb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pfl, o[hb], 0, 0, 0);
      }
    }
  }

  float l_tot = l_run + __shfl_xor(l_run, 16, kWave);
  l_tot += __shfl_xor(l_tot, 32, kWave);
  if (qi < nrows) {
    const int gi = qi / a.R, row = qi % a.R;
    const int h = kvh * grp + gi;
    const int64_t base = ((int64_t)(b * a.n_q + h) * a.R + row) * a.S + blockIdx.y;
    float* op = a.Opart + base * HD;
#pragma unroll
    for (int hb = 0; hb < NHB; ++hb)
      *(float4*)(op + hb * 16 + g4 * 4) = make_float4(o[hb][0], o[hb][1], o[hb][2], o[hb][3]);
    if (g4 == 0) {
      a.MLpart[base * 2] = m_run;
      a.MLpart[base * 2 + 1] = l_tot;
    }
  }
}

// Scalar context pass (float32 model path; any dtype): one wave per (request, head,
// row), lanes own head_dim entries, keys walked in order.  Emits one partial (S == 1).
template <typename T, int HD>
__global__ __launch_bounds__(256) void attn_ctx_scalar(AttnArgs a) {
  constexpr int PER = HD / 64;
  const int wid = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (wid >= a.B * a.n_q * a.R) return;
  const int lane = threadIdx.x & 63;
  const int row = wid % a.R, bh = wid / a.R, h = bh % a.n_q, b = bh / a.n_q;
  const int grp = a.n_q / a.n_kv, kvh = h / grp, gi = h % grp;
  const int L = min(max(a.ctx_len[b], 0), a.cap);
  if (L <= 0) return;
  const T* qp = (const T*)a.Q + (((int64_t)(b * a.n_kv + kvh) * grp + gi) * a.R + row) * HD;
  float q[PER], o[PER];
#pragma unroll
  for (int c = 0; c < PER; ++c) {
    q[c] = ld_f(qp + lane + 64 * c);
    o[c] = 0.f;
  }
  const int64_t kvbase = (int64_t)(b * a.n_kv + kvh);
  const T* Kg = (const T*)a.Kc + kvbase * a.cap * HD;
  const T* Vg = (const T*)a.Vc + kvbase * HD * a.cap;
  const float sc = kLog2e / sqrtf((float)HD);
  float M = -INFINITY, Ls = 0.f;
  for (int key = 0; key < L; ++key) {
    float d = 0.f;
#pragma unroll
    for (int c = 0; c < PER; ++c) d = fmaf(q[c], ld_f(Kg + (int64_t)key * HD + lane + 64 * c), d);
    d = wave_sum(d) * sc;
    const float mn = fmaxf(M, d);
    const float al = exp2f(M - mn), p = exp2f(d - mn);
    Ls = Ls * al + p;
#pragma unroll
    for (int c = 0; c < PER; ++c)
      o[c] = fmaf(p, ld_f(Vg + (int64_t)(lane + 64 * c) * a.cap + key), o[c] * al);
    M = mn;
  }
  const int64_t base = ((int64_t)(b * a.n_q + h) * a.R + row) * a.S;
#pragma unroll
  for (int c = 0; c < PER; ++c) a.Opart[base * HD + lane + 64 * c] = o[c];
  if (lane == 0) {
    a.MLpart[base * 2] = M;
    a.MLpart[base * 2 + 1] = Ls;
  }
}

template <typename T, int HD>
__global__ __launch_bounds__(256) void attn_merge(AttnArgs a) {
  constexpr int PER = HD / 64;
  const int wid = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (wid >= a.B * a.n_q * a.R) return;
  const int lane = threadIdx.x & 63;
  const int row = wid % a.R, bh = wid / a.R, h = bh % a.n_q, b = bh / a.n_q;
  const int grp = a.n_q / a.n_kv, kvh = h / grp, gi = h % grp;
  const T* qp = (const T*)a.Q + (((int64_t)(b * a.n_kv + kvh) * grp + gi) * a.R + row) * HD;
  float q[PER], o[PER];
#pragma unroll
  for (int c = 0; c < PER; ++c) {
    q[c] = ld_f(qp + lane + 64 * c);
    o[c] = 0.f;
  }
  float M = -INFINITY, Ls = 0.f;
  const int L = min(max(a.ctx_len[b], 0), a.cap);
  const int64_t pbase = ((int64_t)(b * a.n_q + h) * a.R + row) * a.S;
  for (int s = 0; s < a.S; ++s) {
    if (s * a.chunk >= L) break;
    const float ms = a.MLpart[(pbase + s) * 2], ls = a.MLpart[(pbase + s) * 2 + 1];
    const float mn = fmaxf(M, ms);
    const float al = exp2f(M - mn), bs = exp2f(ms - mn);
    Ls = Ls * al + ls * bs;
#pragma unroll
    for (int c = 0; c < PER; ++c) o[c] = o[c] * al + a.Opart[(pbase + s) * HD + lane + 64 * c] * bs;
    M = mn;
  }
  // in-block keys under the tree mask
  const int g = a.gamma;
  int n_spine, branch = -1;
  if (row <= g || a.spine_only) {
    n_spine = row + 1;
  } else {
    branch = (row - g - 1) / g;
    n_spine = branch + 1;
  }
  const int64_t kb = (int64_t)(b * a.n_kv + kvh) * a.R;
  const T* Kp = (const T*)a.Kb + kb * HD;
  const T* Vp = (const T*)a.Vb + kb * HD;
  const float sc = kLog2e / sqrtf((float)HD);
  const int n_keys = n_spine + (branch >= 0 ? g : 0);
  for (int t = 0; t < n_keys; ++t) {
    const int key = t < n_spine ? t : g + 1 + branch * g + (t - n_spine);
    float d = 0.f;
#pragma unroll
    for (int c = 0; c < PER; ++c) d = fmaf(q[c], ld_f(Kp + (int64_t)key * HD + lane + 64 * c), d);
    d = wave_sum(d) * sc;
    const float mn = fmaxf(M, d);
    const float al = exp2f(M - mn), p = exp2f(d - mn);
    Ls = Ls * al + p;
#pragma unroll
    for (int c = 0; c < PER; ++c) o[c] = fmaf(p, ld_f(Vp + (int64_t)key * HD + lane + 64 * c), o[c] * al);
    M = mn;
  }
  const float inv = 1.0f / Ls;
  T* op = (T*)a.O + (int64_t)(b * a.R + row) * (a.n_q * HD) + h * HD;
#pragma unroll
  for (int c = 0; c < PER; ++c) st_f(op + lane + 64 * c, o[c] * inv);
}

template <typename T, int HD>
hipError_t run_attention(const AttnArgs& a, hipStream_t st, bool mfma) {
  const int waves = a.B * a.n_q * a.R;
  const int blocks = (waves + 3) / 4;
  {
    Phase ph("attn_ctx", st);
    if (mfma) {
      const int nrows = (a.n_q / a.n_kv) * a.R;
      dim3 grid((nrows + 63) / 64, a.S, a.B * a.n_kv);
      hipLaunchKernelGGL((attn_ctx_mfma<HD>), grid, dim3(256), 0, st, a);
    } else {
      hipLaunchKernelGGL((attn_ctx_scalar<T, HD>), dim3(blocks), dim3(256), 0, st, a);
    }
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  {
    Phase ph("attn_merge", st);
    hipLaunchKernelGGL((attn_merge<T, HD>), dim3(blocks), dim3(256), 0, st, a);
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attention(int dtype, const AttnArgs& a, hipStream_t st) {
  if (dtype == 1) {
    return a.hd == 128 ? run_attention<bf16_t, 128>(a, st, true) : run_attention<bf16_t, 64>(a, st, true);
  }
  return a.hd == 128 ? run_attention<float, 128>(a, st, false) : run_attention<float, 64>(a, st, false);
}

}  // namespace dpara
