// Row assembly, RMSNorm, q/k-norm + RoPE and the context-append kernels.
#include <math.h>

#include <type_traits>

#include "common.h"
#include "internal.h"

namespace dpara {
namespace {

constexpr int kMaxPlanes = 16;  // split-K partial planes a consumer may have to add

// float4 form for the row kernels: planes are loaded in batches of 4 (bounded registers,
// still 4 loads in flight per slot), added in plane order.
__device__ __forceinline__ float4 sum_planes4(float4 acc, const float* p, int64_t stride, int n) {
  for (int s0 = 0; s0 < n; s0 += 4) {
    float4 v[4];
#pragma unroll
    for (int q = 0; q < 4; ++q)
      v[q] = s0 + q < n ? *(const float4*)(p + (s0 + q) * stride) : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int q = 0; q < 4; ++q)
      if (s0 + q < n) {
        acc.x += v[q].x;
        acc.y += v[q].y;
        acc.z += v[q].z;
        acc.w += v[q].w;
      }
  }
  return acc;
}

// Row `row` of request b of the block: spine rows take their token's embedding, mask rows the
// mask embedding.
template <typename T>
__device__ __forceinline__ void assemble_row(int row, int b, int R, int gamma, int H, int V, const int* spine,
                                             const T* embed, const T* mask_emb, float* X, int* status) {
  const T* src = mask_emb;
  if (row <= gamma) {
    int t = spine[b * (gamma + 1) + row];
    if (t < 0 || t >= V) {
      if (threadIdx.x == 0) raise_status(status, 1);
      t = 0;
    }
    src = embed + (int64_t)t * H;
  }
  float* dst = X + ((int64_t)b * R + row) * H;
  // 8 elements (one 16- or 32-byte chunk) per thread and iteration; H % 8 == 0
#pragma unroll 2
  for (int i = threadIdx.x * 8; i < H; i += 256 * 8) {
    float4 lo, hi;
    if constexpr (sizeof(T) == 2) {
      const uint4 u = *(const uint4*)(src + i);
      lo = make_float4(__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xFFFF0000u), __uint_as_float(u.y << 16),
                       __uint_as_float(u.y & 0xFFFF0000u));
      hi = make_float4(__uint_as_float(u.z << 16), __uint_as_float(u.z & 0xFFFF0000u), __uint_as_float(u.w << 16),
                       __uint_as_float(u.w & 0xFFFF0000u));
    } else {
      lo = *(const float4*)(src + i);
      hi = *(const float4*)(src + i + 4);
    }
    *(float4*)(dst + i) = lo;
    *(float4*)(dst + i + 4) = hi;
  }
}

// Four consecutive outputs in one store (8 bytes of bf16, 16 of float32; the address is a
// multiple of 4 elements).
__device__ __forceinline__ void st4(bf16_t* p, float a, float b, float c, float d) {
  *(uint2*)p = make_uint2((uint32_t)f2bf(a) | ((uint32_t)f2bf(b) << 16), (uint32_t)f2bf(c) | ((uint32_t)f2bf(d) << 16));
}
__device__ __forceinline__ void st4(float* p, float a, float b, float c, float d) { *(float4*)p = make_float4(a, b, c, d); }

// One block (8 waves) per output row, VN float4 per thread.  x = X row + the S pending
// split-K partial planes of that row (added in plane order); optionally x is written back
// into X; y = x / rms(x) * g.
constexpr int kNormThreads = 512;
// FRAG: Y is bf16 in MFMA fragment order (frag_index) instead of row-major.
template <typename TO, int VN, int FRAG = 0, int NTH = kNormThreads>
__global__ __launch_bounds__(NTH) void rmsnorm_rows(int H, float* X, int grp, int64_t in_stride,
                                                             int in_off, const float* P, int S, int64_t pstride,
                                                             int write_back, const float* g, float eps, TO* Y) {
  __shared__ float red[NTH / 64];
  const int m = blockIdx.x;
  const int64_t roff = (int64_t)(m / grp) * in_stride + (int64_t)(in_off + m % grp) * H;
  float* x = X + roff;
  float4 v[VN];
  float ss = 0.f;
#pragma unroll
  for (int t = 0; t < VN; ++t) {
    const int i = (threadIdx.x + NTH * t) * 4;
    if (i < H) {
      const float4 a = sum_planes4(*(const float4*)(x + i), P + roff + i, pstride, S);
      if (write_back && S > 0) *(float4*)(x + i) = a;
      v[t] = a;
      ss += a.x * a.x + a.y * a.y + a.z * a.z + a.w * a.w;
    }
  }
  ss = block_sum<NTH / 64>(ss, red);
  const float r = 1.0f / sqrtf(ss / (float)H + eps);
  // fragment blocks: 4 consecutive k of one row stay consecutive (k % 4 == 0), and the 8
  // threads of one 32-k block row write its 64 bytes together
  TO* y = FRAG ? Y : Y + (int64_t)m * H;
#pragma unroll
  for (int t = 0; t < VN; ++t) {
    const int i = (threadIdx.x + NTH * t) * 4;
    if (i < H) {
      const float4 gg = *(const float4*)(g + i);
      st4(FRAG ? Y + frag_index(m, i, H) : y + i, v[t].x * r * gg.x, v[t].y * r * gg.y, v[t].z * r * gg.z,
          v[t].w * r * gg.w);
    }
  }
}

// Entry idx of request b's RoPE table: (cos, sin) of position ctx_len + pos_off + idx / (hd/2).
__device__ __forceinline__ void rope_entry(int b, int idx, int n_pos, int hd, double base, const int* ctx_len,
                                           int pos_off, float2* table) {
  const int half = hd / 2;
  if (idx >= n_pos * half) return;
  const int i = idx / half, p = idx % half;
  float c, s;
  rope_cs(max(ctx_len[b], 0) + pos_off + i, p, hd, base, &c, &s);
  table[((int64_t)b * n_pos + i) * half + p] = make_float2(c, s);
}

__global__ void rope_table_kernel(int n_pos, int hd, double base, const int* ctx_len, int pos_off,
                                  float2* table) {
  rope_entry(blockIdx.y, blockIdx.x * blockDim.x + threadIdx.x, n_pos, hd, base, ctx_len, pos_off, table);
}

// The backbone's first two steps in one launch: blocks x < R assemble rows, the blocks past R
// fill the RoPE table (256 entries each).
template <typename T>
__global__ __launch_bounds__(256) void assemble_rows_rope(int R, int gamma, int H, int V, const int* spine,
                                                          const T* embed, const T* mask_emb, float* X, int* status,
                                                          int n_pos, int hd, double base, const int* ctx_len,
                                                          float2* table) {
  if ((int)blockIdx.x < R)
    assemble_row(blockIdx.x, blockIdx.y, R, gamma, H, V, spine, embed, mask_emb, X, status);
  else
    rope_entry(blockIdx.y, ((int)blockIdx.x - R) * 256 + threadIdx.x, n_pos, hd, base, ctx_len, 0, table);
}

// Grid (head-slot groups, rows): HD/4 lanes per (row, head slot), 4 consecutive entries per
// lane, so a wave covers 64 / (HD/4) slots; the slots are the q heads, then the k heads, then
// the v heads of the fused QKV row, summed over the S split-K planes (in plane order).  The
// rotate-half partner of a lane's entries sits HD/8 lanes away in the same group.
// In-block keys are stored [Rp][hd] and values transposed [hd][Rp] per request and KV head
// (Rp = R rounded up to 64 keys) for the MFMA attention pass.
template <typename T, int HD>
__global__ __launch_bounds__(256) void qk_norm_rope(int R, int Rp, int gamma, int n_q, int n_kv, int qk_norm,
                                                    float eps, const float* QKV, int S, int64_t pstride,
                                                    const float* qn, const float* kn, const float2* table, T* Q,
                                                    T* Kb, T* Vb) {
  constexpr int LPS = HD / 4, SPW = 64 / LPS, HALF = HD / 2;
  const int m = blockIdx.y;
  const int b = m / R, row = m % R;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int sl = lane % LPS, j0 = sl * 4;
  const int slot = (blockIdx.x * 4 + wave) * SPW + lane / LPS;
  const int grp = n_q / n_kv, n_slots = n_q + 2 * n_kv;
  const bool valid = slot < n_slots;
  const float* x = QKV + ((int64_t)m * n_slots + (valid ? slot : 0)) * HD + j0;
  float4 pv[kMaxPlanes];
#pragma unroll
  for (int s = 0; s < kMaxPlanes; ++s)
    pv[s] = (valid && s < S) ? *(const float4*)(x + s * pstride) : make_float4(0.f, 0.f, 0.f, 0.f);
  float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
  for (int s = 0; s < kMaxPlanes; ++s)
    if (s < S) {
      v.x += pv[s].x;
      v.y += pv[s].y;
      v.z += pv[s].z;
      v.w += pv[s].w;
    }
  if (slot >= n_q + n_kv) {  // values (or past the last slot): transposed store [hd][Rp]
    if (!valid) return;
    const int kvh = slot - n_q - n_kv;
    T* dst = Vb + ((int64_t)(b * n_kv + kvh) * HD + j0) * Rp + row;
    st_f(dst, v.x);
    st_f(dst + Rp, v.y);
    st_f(dst + 2 * Rp, v.z);
    st_f(dst + 3 * (int64_t)Rp, v.w);
    return;
  }
  // q/k slots: whole lane groups take this branch together (the v slots follow them)
  const bool isq = slot < n_q;
  if (qk_norm) {
    float ss = v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
#pragma unroll
    for (int o = LPS / 2; o > 0; o >>= 1) ss += __shfl_xor(ss, o, 64);
    const float r = 1.0f / sqrtf(ss / (float)HD + eps);
    const float4 gg = *(const float4*)((isq ? qn : kn) + j0);
    v.x = v.x * r * gg.x;
    v.y = v.y * r * gg.y;
    v.z = v.z * r * gg.z;
    v.w = v.w * r * gg.w;
  }
  float4 pr;  // the rotate-half partner entries
  pr.x = __shfl_xor(v.x, LPS / 2, 64);
  pr.y = __shfl_xor(v.y, LPS / 2, 64);
  pr.z = __shfl_xor(v.z, LPS / 2, 64);
  pr.w = __shfl_xor(v.w, LPS / 2, 64);
  const bool first = j0 < HALF;
  const float2* cs = table + ((int64_t)b * (2 * gamma + 1) + row_pos_offset(row, gamma)) * HALF + (j0 % HALF);
  const float2 c0 = cs[0], c1 = cs[1], c2 = cs[2], c3 = cs[3];
  // first half: y = x cos - x' sin; second half: y = x cos + x' sin (x' = the partner entry)
  const float sg = first ? -1.f : 1.f;
  const float y0 = v.x * c0.x + sg * pr.x * c0.y;
  const float y1 = v.y * c1.x + sg * pr.y * c1.y;
  const float y2 = v.z * c2.x + sg * pr.z * c2.y;
  const float y3 = v.w * c3.x + sg * pr.w * c3.y;
  if (!valid) return;
  T* dst;
  if (isq) {
    const int kvh = slot / grp, gi = slot % grp;
    dst = Q + (((int64_t)(b * n_kv + kvh) * grp + gi) * R + row) * HD + j0;
  } else {
    const int kvh = slot - n_q;
    dst = Kb + ((int64_t)(b * n_kv + kvh) * Rp + row) * HD + j0;
  }
  st4(dst, y0, y1, y2, y3);
}

template <typename T>
__global__ __launch_bounds__(256) void gather_feats(int CH, int c0, int n_max, int H, const T* feats, T* F) {
  const int m = blockIdx.x, b = m / CH, i = m % CH;
  const int c = c0 + i;
  // 16-byte chunks; H * sizeof(T) % 16 == 0
  uint4* dst = (uint4*)(F + (int64_t)m * H);
  const int nch = H * (int)sizeof(T) / 16;
  if (c >= n_max) {
    for (int k = threadIdx.x; k < nch; k += 256) dst[k] = make_uint4(0, 0, 0, 0);
    return;
  }
  const uint4* src = (const uint4*)(feats + ((int64_t)b * n_max + c) * H);
#pragma unroll 4
  for (int k = threadIdx.x; k < nch; k += 256) dst[k] = src[k];
}

__device__ __forceinline__ int clamp_count(int n, int n_max) { return n < 0 ? 0 : (n > n_max ? n_max : n); }

// K/V of appended rows: k = RoPE(kNorm(W_k f)) at its position, v = W_v f; K rows go to
// [pos][hd], V to the transposed cache [hd][pos].
// Grid (kv-head groups of 4, rows, layers).
template <typename T>
__global__ __launch_bounds__(256) void kv_store(int CH, int c0, int n_max, int n_kv, int hd, int qk_norm, float eps,
                                                const float2* rope, const float* KV, int S, int64_t pstride,
                                                KvLayers kls, const int* n_new, const int* ctx_len, int cap,
                                                T* Kc, T* Vc, int64_t layer_elems) {
  const int m = blockIdx.y, b = m / CH, i = m % CH, l = blockIdx.z, nl = gridDim.z;
  const int c = c0 + i;
  if (c >= clamp_count(n_new[b], n_max)) return;
  const int pos = max(ctx_len[b], 0) + c;
  if (pos >= cap) return;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int half = hd / 2;
  const float* kn = kls.kn[l];
  Kc += l * layer_elems;
  Vc += l * layer_elems;
  const float* src = KV + ((int64_t)m * nl + l) * 2 * n_kv * hd;
  const int kvh = blockIdx.x * 4 + wave;  // one wave per (row, kv head)
  if (kvh >= n_kv) return;
  const float* x = src + kvh * hd;
  const float* xv = src + (n_kv + kvh) * hd;
  const bool act = lane < half;
  // every plane of the row's K pair and V entries is requested before any is summed
  float pk1[kMaxPlanes], pk2[kMaxPlanes], pv[2][kMaxPlanes];
#pragma unroll
  for (int s = 0; s < kMaxPlanes; ++s) {
    const bool on = s < S;
    pk1[s] = on && act ? x[s * pstride + lane] : 0.f;
    pk2[s] = on && act ? x[s * pstride + lane + half] : 0.f;
#pragma unroll
    for (int q = 0; q < 2; ++q) pv[q][s] = on && lane + 64 * q < hd ? xv[s * pstride + lane + 64 * q] : 0.f;
  }
  float x1 = 0.f, x2 = 0.f, v[2] = {0.f, 0.f};
#pragma unroll
  for (int s = 0; s < kMaxPlanes; ++s) {
    if (s < S) {
      x1 += pk1[s];
      x2 += pk2[s];
      v[0] += pv[0][s];
      v[1] += pv[1][s];
    }
  }
  if (qk_norm) {
    const float ss = wave_sum(x1 * x1 + x2 * x2);
    const float r = 1.0f / sqrtf(ss / (float)hd + eps);
    if (act) {
      x1 = x1 * r * kn[lane];
      x2 = x2 * r * kn[lane + half];
    }
  }
  const int64_t kvb = (int64_t)(b * n_kv + kvh);
  if (act) {
    const float2 cs = rope[(int64_t)m * half + lane];  // row m of this chunk, position pos
    T* kd = Kc + (kvb * cap + pos) * hd;
    st_f(kd + lane, x1 * cs.x - x2 * cs.y);
    st_f(kd + lane + half, x2 * cs.x + x1 * cs.y);
  }
#pragma unroll
  for (int q = 0; q < 2; ++q)
    if (lane + 64 * q < hd) st_f(Vc + (kvb * hd + lane + 64 * q) * cap + pos, v[q]);
}

// Hidden state of every row after a layer: bf16(X + the S pending split-K planes), written
// to out[m * n_out + j] (rows of H entries), 4 entries per thread.
template <typename TO>
__global__ __launch_bounds__(256) void emit_hidden(int H, const float* X, const float* P, int S, int64_t pstride,
                                                   TO* out, int n_out, int j) {
  const int m = blockIdx.y;
  const int i = (blockIdx.x * 256 + threadIdx.x) * 4;
  if (i >= H) return;
  float4 v = *(const float4*)(X + (int64_t)m * H + i);
  for (int s = 0; s < S; ++s) {
    const float4 q = *(const float4*)(P + s * pstride + (int64_t)m * H + i);
    v.x += q.x;
    v.y += q.y;
    v.z += q.z;
    v.w += q.w;
  }
  TO* o = out + ((int64_t)m * n_out + j) * H + i;
  if constexpr (sizeof(TO) == 4) {
    *(float4*)o = v;
  } else {
    *(uint2*)o = make_uint2(f2bf(v.x) | ((uint32_t)f2bf(v.y) << 16), f2bf(v.z) | ((uint32_t)f2bf(v.w) << 16));
  }
}

__global__ void ctx_len_update_kernel(int B, int n_max, int cap, const int* n_new, int* ctx_len, int* status) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= B) return;
  const int raw = n_new[b];
  const int n = clamp_count(raw, n_max);
  if (n != raw) raise_status(status, 8);
  int L = max(ctx_len[b], 0) + n;
  if (L > cap) {
    raise_status(status, 2);
    L = cap;
  }
  ctx_len[b] = L;
}

__global__ void clear_status_kernel(int* status) { status[threadIdx.x] = 0; }

}  // namespace

template <typename TO, int VN>
void rmsnorm_launch(int rows, int H, float* X, int grp, int64_t in_stride, int in_off, const float* P, int S,
                    int64_t pstride, int write_back, const float* g, float eps, void* Y, hipStream_t st) {
  // Up to 64 rows (a target verifying 17 rows a request) each row's workgroup is one of only a
  // few on the chip: 1024 threads per row put twice the loads in flight on its CU.
  if (rows <= 64 && (H / 4 + 1023) / 1024 <= (VN + 1) / 2) {
    hipLaunchKernelGGL((rmsnorm_rows<TO, (VN + 1) / 2, 0, 1024>), dim3(rows), dim3(1024), 0, st, H, X, grp, in_stride,
                       in_off, P, S, pstride, write_back, g, eps, (TO*)Y);
    return;
  }
  hipLaunchKernelGGL((rmsnorm_rows<TO, VN>), dim3(rows), dim3(kNormThreads), 0, st, H, X, grp, in_stride, in_off, P,
                     S, pstride, write_back, g, eps, (TO*)Y);
}

template <typename TO>
hipError_t rmsnorm_dispatch(int rows, int H, float* X, int grp, int64_t in_stride, int in_off, const float* P,
                            int S, int64_t pstride, int write_back, const float* g, float eps, void* Y,
                            hipStream_t st) {
  const int vn = (H / 4 + kNormThreads - 1) / kNormThreads;
  switch (vn) {
    case 1: rmsnorm_launch<TO, 1>(rows, H, X, grp, in_stride, in_off, P, S, pstride, write_back, g, eps, Y, st); break;
    case 2: rmsnorm_launch<TO, 2>(rows, H, X, grp, in_stride, in_off, P, S, pstride, write_back, g, eps, Y, st); break;
    case 3: rmsnorm_launch<TO, 3>(rows, H, X, grp, in_stride, in_off, P, S, pstride, write_back, g, eps, Y, st); break;
    case 4: rmsnorm_launch<TO, 4>(rows, H, X, grp, in_stride, in_off, P, S, pstride, write_back, g, eps, Y, st); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_rmsnorm(int out_dtype, int rows, int H, float* X, int grp, int64_t in_stride, int in_off,
                          const float* P, int S, int64_t pstride, int write_back, const float* g, float eps,
                          void* Y, hipStream_t st) {
  if (rows <= 0) return hipSuccess;
  if (H > 16 * kNormThreads || H % 4 || S < 0 || S > kMaxPlanes) return hipErrorInvalidValue;
  if (out_dtype == 1)
    return rmsnorm_dispatch<bf16_t>(rows, H, X, grp, in_stride, in_off, P, S, pstride, write_back, g, eps, Y, st);
  return rmsnorm_dispatch<float>(rows, H, X, grp, in_stride, in_off, P, S, pstride, write_back, g, eps, Y, st);
}

hipError_t launch_rmsnorm_frag(int rows, int H, float* X, const float* P, int S, int64_t pstride,
                               const float* g, float eps, void* Y, hipStream_t st) {
  if (rows <= 0) return hipSuccess;
  if (H > 16 * kNormThreads || H % 32 || S < 0 || S > kMaxPlanes) return hipErrorInvalidValue;
  const int vn = (H / 4 + kNormThreads - 1) / kNormThreads;
  auto go = [&](auto kern) {
    hipLaunchKernelGGL(kern, dim3(rows), dim3(kNormThreads), 0, st, H, X, rows, (int64_t)0, 0, P, S, pstride, 1, g,
                       eps, (bf16_t*)Y);
    return hipGetLastError();
  };
  switch (vn) {
    case 1: return go(rmsnorm_rows<bf16_t, 1, 1>);
    case 2: return go(rmsnorm_rows<bf16_t, 2, 1>);
    case 3: return go(rmsnorm_rows<bf16_t, 3, 1>);
    case 4: return go(rmsnorm_rows<bf16_t, 4, 1>);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_assemble_rows_rope(int dtype, int B, int R, int gamma, int H, int V, const int* spine,
                                     const void* embed, const void* mask_emb, float* X, int* status, int n_pos,
                                     int hd, float base, const int* ctx_len, float2* table, hipStream_t st) {
  dim3 grid(R + (n_pos * (hd / 2) + 255) / 256, B);
  if (dtype == 1)
    hipLaunchKernelGGL(assemble_rows_rope<bf16_t>, grid, dim3(256), 0, st, R, gamma, H, V, spine,
                       (const bf16_t*)embed, (const bf16_t*)mask_emb, X, status, n_pos, hd, (double)base, ctx_len,
                       table);
  else
    hipLaunchKernelGGL(assemble_rows_rope<float>, grid, dim3(256), 0, st, R, gamma, H, V, spine,
                       (const float*)embed, (const float*)mask_emb, X, status, n_pos, hd, (double)base, ctx_len,
                       table);
  return hipGetLastError();
}

hipError_t launch_rope_table(int B, int n_pos, int hd, float base, const int* ctx_len, int pos_off,
                             float2* table, hipStream_t st) {
  const int n = n_pos * (hd / 2);
  dim3 grid((n + 255) / 256, B);
  hipLaunchKernelGGL(rope_table_kernel, grid, dim3(256), 0, st, n_pos, hd, (double)base, ctx_len, pos_off,
                     table);
  return hipGetLastError();
}

hipError_t launch_qk_norm_rope(int dtype, int B, int R, int Rp, int gamma, int n_q, int n_kv, int hd, int qk_norm,
                               float eps, const float* QKV, int S, const float* qn, const float* kn,
                               const float2* table, void* Q, void* Kb, void* Vb, hipStream_t st) {
  if (Rp < R || S < 1 || S > kMaxPlanes || (hd != 64 && hd != 128)) return hipErrorInvalidValue;
  const int n_slots = n_q + 2 * n_kv, per_block = 4 * (256 / hd);
  dim3 grid((n_slots + per_block - 1) / per_block, B * R);
  const int64_t pstride = (int64_t)B * R * n_slots * hd;
  auto go = [&](auto kern, auto* q) {
    using TT = std::remove_pointer_t<decltype(q)>;
    hipLaunchKernelGGL(kern, grid, dim3(256), 0, st, R, Rp, gamma, n_q, n_kv, qk_norm, eps, QKV, S, pstride, qn, kn,
                       table, (TT*)Q, (TT*)Kb, (TT*)Vb);
    return hipGetLastError();
  };
  if (dtype == 1)
    return hd == 128 ? go(qk_norm_rope<bf16_t, 128>, (bf16_t*)nullptr) : go(qk_norm_rope<bf16_t, 64>, (bf16_t*)nullptr);
  return hd == 128 ? go(qk_norm_rope<float, 128>, (float*)nullptr) : go(qk_norm_rope<float, 64>, (float*)nullptr);
}

hipError_t launch_gather_feats(int dtype, int B, int CH, int c0, int n_max, int H, const void* feats,
                               void* F, hipStream_t st) {
  if (dtype == 1)
    hipLaunchKernelGGL(gather_feats<bf16_t>, dim3(B * CH), dim3(256), 0, st, CH, c0, n_max, H,
                       (const bf16_t*)feats, (bf16_t*)F);
  else
    hipLaunchKernelGGL(gather_feats<float>, dim3(B * CH), dim3(256), 0, st, CH, c0, n_max, H,
                       (const float*)feats, (float*)F);
  return hipGetLastError();
}

hipError_t launch_kv_store(int dtype, int B, int CH, int c0, int n_max, int n_kv, int hd, int qk_norm,
                           float eps, const float2* rope, const float* KV, int S, int nl, const KvLayers& kn,
                           const int* n_new, const int* ctx_len, int cap, void* Kc, void* Vc, size_t layer_elems,
                           int* status, hipStream_t st) {
  (void)status;
  if (S < 1 || S > kMaxPlanes || nl < 1 || nl > kMaxAppendLayers) return hipErrorInvalidValue;
  const int64_t pstride = (int64_t)B * CH * nl * 2 * n_kv * hd;
  const dim3 grid((n_kv + 3) / 4, B * CH, nl);
  if (dtype == 1)
    hipLaunchKernelGGL(kv_store<bf16_t>, grid, dim3(256), 0, st, CH, c0, n_max, n_kv, hd, qk_norm, eps,
                       rope, KV, S, pstride, kn, n_new, ctx_len, cap, (bf16_t*)Kc, (bf16_t*)Vc,
                       (int64_t)layer_elems);
  else
    hipLaunchKernelGGL(kv_store<float>, grid, dim3(256), 0, st, CH, c0, n_max, n_kv, hd, qk_norm, eps,
                       rope, KV, S, pstride, kn, n_new, ctx_len, cap, (float*)Kc, (float*)Vc,
                       (int64_t)layer_elems);
  return hipGetLastError();
}

hipError_t launch_emit_hidden(int rows, int H, const float* X, const float* P, int S, int64_t pstride, void* out,
                              int n_out, int j, hipStream_t st, int out_f32) {
  if (rows <= 0) return hipSuccess;
  if (H % 4 || S < 0 || S > kMaxPlanes || j < 0 || j >= n_out) return hipErrorInvalidValue;
  const dim3 grid((H / 4 + 255) / 256, rows);
  if (out_f32)
    hipLaunchKernelGGL(emit_hidden<float>, grid, dim3(256), 0, st, H, X, P, S, pstride, (float*)out, n_out, j);
  else
    hipLaunchKernelGGL(emit_hidden<bf16_t>, grid, dim3(256), 0, st, H, X, P, S, pstride, (bf16_t*)out, n_out, j);
  return hipGetLastError();
}

hipError_t launch_ctx_len_update(int B, int n_max, int cap, const int* n_new, int* ctx_len, int* status,
                                 hipStream_t st) {
  hipLaunchKernelGGL(ctx_len_update_kernel, dim3((B + 63) / 64), dim3(64), 0, st, B, n_max, cap, n_new, ctx_len,
                     status);
  return hipGetLastError();
}

hipError_t launch_clear_status(int* status, hipStream_t st) {
  hipLaunchKernelGGL(clear_status_kernel, dim3(1), dim3(1), 0, st, status);
  return hipGetLastError();
}

}  // namespace dpara
