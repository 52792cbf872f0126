// Multi-boundary attention of the all-boundary backbone (tree mask of Section 3.2).
//
// Each request's (gamma+1)^2 block rows see the whole cached context plus, under the tree
// mask, some of the block's own keys: spine t_j sees t_0..t_j, branch r's mask rows see
// t_0..t_r and all of branch r's masks.  For one request and KV head the keys therefore
// form one virtual sequence: ceil(L/64) blocks of context followed by ceil(R/64) blocks of
// in-block keys (dense, masked per element).  Workgroups split that sequence evenly.
//
// bf16 path (attn_mfma): one workgroup = 8 waves x 16 query rows (all query heads of the
// KV group share the keys) over a contiguous range of 64-key blocks.  K (keys x head_dim)
// and V^T (head_dim x keys; both the cache and the in-block values are stored transposed)
// stream through a double-buffered, XOR-swizzled LDS ring filled by direct global->LDS DMA:
// the next block's DMA is issued before the current block's MFMAs, so its latency hides
// behind the math.  S^T = K Q^T and O^T += V^T P^T use v_mfma_f32_16x16x32_bf16 with an
// online softmax in log2 units.  The K operand rows are permuted so that each
// lane's probabilities form 8 consecutive keys, which makes every V^T operand one
// 16-byte LDS read.  P enters the PV product as a bf16 hi + lo pair (two MFMAs), so the
// probabilities keep ~16 significant bits: a single bf16 rounding of P moves the result
// by about one bf16 ulp of the hidden state, which is as large as the whole error budget.
// With one workgroup per row tile (S == 1) the kernel normalises and writes O itself;
// otherwise each writes an unnormalised partial (O, m, l) and attn_fold combines them.
#include <math.h>

#include <type_traits>

#include "common.h"
#include "internal.h"

namespace dpara {
namespace {

constexpr float kLog2e = 1.4426950408889634f;
#ifndef DPARA_ATTN_WAVES
#define DPARA_ATTN_WAVES 8
#endif
#ifndef DPARA_ATTN_TILES
#define DPARA_ATTN_TILES 1
#endif
#ifndef DPARA_ATTN_STAGES
#define DPARA_ATTN_STAGES 2
#endif
constexpr int kKeyBlock = 64;
constexpr int kAttnWaves = DPARA_ATTN_WAVES;   // waves per workgroup
constexpr int kAttnTiles = DPARA_ATTN_TILES;   // 16-row query tiles per wave
constexpr int kAttnStages = DPARA_ATTN_STAGES; // LDS ring depth
constexpr int kRowsPerWG = kAttnWaves * kAttnTiles * 16;

// LDS swizzles (16-byte chunk index within a row).  K rows hold head_dim entries; a K
// operand read has 16 lanes on rows whose index bits 0,1,3,4 vary (bit 2 fixed), V^T
// rows hold 64 keys (128 bytes) and a read has 16 lanes on 16 consecutive rows.
template <int HD>
__device__ __forceinline__ int k_swz(int r, int c) {
  if constexpr (HD == 128) return c ^ ((r & 3) | ((r >> 1) & 12));
  else return c ^ (((r >> 1) & 1) | ((r >> 2) & 6));
}
__device__ __forceinline__ int v_swz(int r, int c) { return c ^ ((r >> 1) & 7); }

__device__ __forceinline__ int grp_rows(const AttnArgs& a) { return (a.n_q / a.n_kv) * a.R; }

// Key offset within a 64-key block held by S^T row i of 16-key MFMA block kb.
__device__ __forceinline__ int key_perm(int kb, int i) { return (kb >> 1) * 32 + (i >> 2) * 8 + (kb & 1) * 4 + (i & 3); }

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

// Maximum and sum over the four 16-lane rows of a wave (lanes lq, lq + 16, lq + 32, lq + 48):
// v_permlane16_swap / v_permlane32_swap exchange whole rows between two registers on the
// VALU, so the reduction needs no LDS round trip.
__device__ __forceinline__ float rows4_max(float x) {
  const uint32_t u = __float_as_uint(x);
  const auto a = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  const float y = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const uint32_t v = __float_as_uint(y);
  const auto b = __builtin_amdgcn_permlane32_swap(v, v, false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ __forceinline__ float rows4_sum(float x) {
  const uint32_t u = __float_as_uint(x);
  const auto a = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  const float y = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  const uint32_t v = __float_as_uint(y);
  const auto b = __builtin_amdgcn_permlane32_swap(v, v, false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

// The running maximum of a row is the reference of its probabilities p = 2^(s - m).  It
// moves only when a block's maximum passes it by more than kLazyMax (log2 units), so the
// accumulators are rescaled rarely; p then stays below 2^kLazyMax, which the bf16 hi + lo
// pair and the float32 sums carry with unchanged relative precision.
constexpr float kLazyMax = 8.f;

__device__ __forceinline__ bf16x8_t as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8_t, v); }

// The K and V^T tiles of a 64-key block are filled by direct global->LDS DMA
// (global_load_lds_dwordx4: lane i's 16 bytes land at M0 + 16*i), through a ring of
// STAGES stages: STAGES-1 blocks are in flight while one is consumed.  Every load is a
// full 16-byte chunk: the context cache and the in-block buffers hold a multiple of 64
// keys, so a block never reads past its buffer; keys past the valid count are excluded
// from the scores by the mask, and their V^T entries are zeroed in LDS (a tail block
// only) so that stale memory cannot turn 0 * V into NaN.
//
// Workgroup = NW waves x U 16-row query tiles per wave.  Fragment reads: the K operand
// row of MFMA block kb for lane lq is key_perm(kb, lq), whose swizzle depends on lq only
// (kb moves bits 2 and 5 of the row, which the swizzle ignores), and the V^T operand row
// hb*16 + lq likewise swizzles by lq only; so each read is a per-lane base plus a
// compile-time offset.
template <int HD, int NW, int U, int STAGES>
__global__ __launch_bounds__(64 * NW) void attn_mfma(AttnArgs a) {
  constexpr int NKS = HD / 32;                 // k-steps over head_dim for S
  constexpr int NHB = HD / 16;                 // 16-row blocks of head_dim for O^T
  constexpr int K_BYTES = kKeyBlock * HD * 2;  // K tile
  constexpr int STAGE_BYTES = 2 * K_BYTES;     // K tile + V^T tile (same size)
  constexpr int NINS = K_BYTES / 1024 / NW;    // DMA instructions per wave per tile
  constexpr int ROWS_WG = NW * U * 16;
  static_assert(NINS * 1024 * NW == K_BYTES, "tile must split evenly over the waves");
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];

  // XCD-aware order: workgroups are dispatched round-robin over the 8 XCDs, so physical id p
  // maps to logical id lid with each XCD taking a contiguous range of lid; row tiles run
  // fastest in lid, so the tiles that read the same key blocks share one XCD's L2.  KV heads
  // are the slowest index, so an XCD's range holds the same heads of every request (with 8 KV
  // heads, one head each) and the XCDs get equal shares of a batch of mixed context lengths;
  // within it the requests come longest context first, so the short ones fill the last round.
  const int n_tiles = (grp_rows(a) + ROWS_WG - 1) / ROWS_WG;
  const int total = n_tiles * a.S * a.B * a.n_kv;
  const int p = blockIdx.x, per_xcd = total >> 3;
  const int lid = p < (per_xcd << 3) ? (p & 7) * per_xcd + (p >> 3) : p;
  const int tile = lid % n_tiles, split = (lid / n_tiles) % a.S, hb = lid / (n_tiles * a.S);
  const int kvh = hb / a.B, rank = hb % a.B;
  int b = rank;
  if (a.B > 1 && a.B <= 64) {
    // the request of this rank by (context length descending, index ascending): lane t ranks
    // request t, every wave the same (no barrier), and the ballot picks the one lane
    const int t = threadIdx.x & 63;
    const int Lt = t < a.B ? min(max(a.ctx_len[t], 0), a.cap) : -1;
    int r = 0;
    for (int u = 0; u < a.B; ++u) {
      const int Lu = min(max(a.ctx_len[u], 0), a.cap);
      r += (Lu > Lt) | ((Lu == Lt) & (u < t));
    }
    b = __builtin_ctzll(__ballot(t < a.B && r == rank));
  }
  const int grp = a.n_q / a.n_kv;
  const int nrows = grp * a.R;
  const int L = min(max(a.ctx_len[b], 0), a.cap);
  const int nb_ctx = (L + kKeyBlock - 1) / kKeyBlock;
  const int nb = nb_ctx + (a.R + kKeyBlock - 1) / kKeyBlock;
  const int per = (nb + a.S - 1) / a.S;
  const int vb_begin = min(nb, split * per);
  const int n_blk = min(nb, vb_begin + per) - vb_begin;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int lq = lane & 15, g4 = lane >> 4;
  const int qrow0 = tile * ROWS_WG + wave * U * 16;
  const bool wave_live = qrow0 < nrows;

  const int64_t kvbase = (int64_t)(b * a.n_kv + kvh);
  const bf16_t* Kg = (const bf16_t*)a.Kc + kvbase * a.cap * HD;
  const bf16_t* Vg = (const bf16_t*)a.Vc + kvbase * HD * a.cap;
  const bf16_t* Kin = (const bf16_t*)a.Kb + kvbase * a.Rp * HD;
  const bf16_t* Vin = (const bf16_t*)a.Vb + kvbase * HD * a.Rp;
  // Per-lane byte offsets of this wave's DMA chunks within a block (instruction j fills tile
  // chunks (wave + NW*j)*64 + lane of K and of V^T); the block's base address is uniform.
  int koff[NINS], voff_ctx[NINS], voff_in[NINS];
#pragma unroll
  for (int j = 0; j < NINS; ++j) {
    const int idx = (wave + NW * j) * 64 + lane;
    const int r = idx / (HD / 8), c = idx % (HD / 8);
    koff[j] = (r * HD + k_swz<HD>(r, c) * 8) * 2;
    const int d = idx / (kKeyBlock / 8), cv = idx % (kKeyBlock / 8);
    voff_ctx[j] = (d * a.cap + v_swz(d, cv) * 8) * 2;
    voff_in[j] = (d * a.Rp + v_swz(d, cv) * 8) * 2;
  }
  auto issue = [&](int vb, int stage) {
    const bool inblk = vb >= nb_ctx;
    const int kb0 = (inblk ? vb - nb_ctx : vb) * kKeyBlock;
    const char* Ks = (const char*)((inblk ? Kin : Kg) + (int64_t)kb0 * HD);
    const char* Vs = (const char*)((inblk ? Vin : Vg) + kb0);
    unsigned char* sb = smem + stage * STAGE_BYTES;
#pragma unroll
    for (int j = 0; j < NINS; ++j)
      __builtin_amdgcn_global_load_lds((const void*)(Ks + koff[j]), (lds_void_t*)(sb + (wave + NW * j) * 1024), 16,
                                       0, 0);
#pragma unroll
    for (int j = 0; j < NINS; ++j)
      __builtin_amdgcn_global_load_lds((const void*)(Vs + (inblk ? voff_in[j] : voff_ctx[j])),
                                       (lds_void_t*)(sb + K_BYTES + (wave + NW * j) * 1024), 16, 0, 0);
  };
  debug_poison_lds<STAGES * STAGE_BYTES>(smem);
#pragma unroll
  for (int st = 0; st < STAGES - 1; ++st)
    if (st < n_blk) issue(vb_begin + st, st);

  // Query fragments (B operand of S^T = K Q^T) and the tree-mask intervals of each row:
  // an in-block key j is visible iff j < e1 or lo2 <= j < lo2 + span.
  const bf16_t* Qp = (const bf16_t*)a.Q + kvbase * nrows * HD;
  bf16x8_t qf[U][NKS];
  int qi[U], e1[U], lo2[U], span[U];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    qi[u] = qrow0 + u * 16 + lq;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks)
      qf[u][ks] = qi[u] < nrows ? *(const bf16x8_t*)(Qp + (int64_t)qi[u] * HD + ks * 32 + g4 * 8)
                                : bf16x8_t{0, 0, 0, 0, 0, 0, 0, 0};
    const int row = qi[u] % a.R, g = a.gamma;
    if (a.spine_only || row <= g) {
      e1[u] = row + 1;
      lo2[u] = span[u] = 0;
    } else {
      const int br = (row - g - 1) / g;
      e1[u] = br + 1;
      lo2[u] = g + 1 + br * g;
      span[u] = g;
    }
  }
  // per-lane LDS byte offsets of the fragment reads within a stage
  const int kx = k_swz<HD>(key_perm(0, lq), 0);
  const int k_lane = key_perm(0, lq) * HD * 2;
  const int v_lane = lq * kKeyBlock * 2;
  const int vx = v_swz(lq, 0);

  f32x4_t o[U][NHB];
#pragma unroll
  for (int u = 0; u < U; ++u)
#pragma unroll
    for (int hb = 0; hb < NHB; ++hb) o[u][hb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  float m_run[U], l_run[U];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    m_run[u] = -INFINITY;
    l_run[u] = 0.f;
  }
  const float sc = kLog2e / sqrtf((float)HD);

  for (int i = 0; i < n_blk; ++i) {
    if (i + STAGES - 2 < n_blk) wait_vmcnt<(STAGES - 2) * 2 * NINS>();
    else wait_vmcnt<0>();
    __builtin_amdgcn_s_barrier();
    if (i + STAGES - 1 < n_blk) issue(vb_begin + i + STAGES - 1, (i + STAGES - 1) % STAGES);
    const unsigned char* sb = smem + (i % STAGES) * STAGE_BYTES;
    const int vb = vb_begin + i;
    const bool inblk = vb >= nb_ctx;
    const int kb0 = (inblk ? vb - nb_ctx : vb) * kKeyBlock;
    const int kend = inblk ? a.R : L;
    if (kb0 + kKeyBlock > kend) {
      // A tail block (at most two per workgroup, a uniform branch): zero the V^T entries of
      // keys >= kend in LDS, so that stale memory past the valid keys cannot turn 0 * V into
      // NaN, and every block then takes the same PV code (one PV path keeps the accumulators
      // in one set of registers: 116 VGPRs, two workgroups per CU).  Thread t owns the CPT
      // consecutive 16-byte chunks from t * CPT of the tile (8 chunks a V^T row).
      static_assert((HD * 8) % (NW * 64) == 0, "the V^T tile's chunks split evenly over the threads");
      constexpr int CPT = HD * 8 / (NW * 64);  // chunks per thread
      unsigned char* vt = smem + (i % STAGES) * STAGE_BYTES + K_BYTES;
#pragma unroll
      for (int q = 0; q < CPT; ++q) {
        const int e = threadIdx.x * CPT + q;  // chunk e of the tile: row e / 8, chunk e % 8
        const int d = e >> 3, c = e & 7;
        const int nv = kend - (kb0 + c * 8);  // valid keys in this chunk (may be <= 0 or >= 8)
        if (nv < 8) {
          uint4* cp = (uint4*)(vt + d * kKeyBlock * 2 + v_swz(d, c) * 16);
          uint4 x = *cp;
          x.x &= (0 < nv ? 0xFFFFu : 0u) | (1 < nv ? 0xFFFF0000u : 0u);
          x.y &= (2 < nv ? 0xFFFFu : 0u) | (3 < nv ? 0xFFFF0000u : 0u);
          x.z &= (4 < nv ? 0xFFFFu : 0u) | (5 < nv ? 0xFFFF0000u : 0u);
          x.w &= (6 < nv ? 0xFFFFu : 0u) | (7 < nv ? 0xFFFF0000u : 0u);
          *cp = x;
        }
      }
      __syncthreads();
    }
    if (!wave_live) continue;
    if (inblk) {
      // Under the tree mask a row sees at most two short runs of in-block keys (the spine
      // prefix and its own branch): a block that none of the wave's rows sees adds nothing
      // (every p is 0, no maximum moves), so the wave skips its products.
      bool need = false;
#pragma unroll
      for (int u = 0; u < U; ++u)
        need |= (kb0 < e1[u]) | ((span[u] > 0) & (kb0 < lo2[u] + span[u]) & (kb0 + kKeyBlock > lo2[u]));
      if (!__any(need)) continue;
    }

    // S^T blocks: s[u][kb][r] = score(key kb0 + key_perm(kb, 4*g4 + r), query qi[u])
    f32x4_t s[U][4];
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) s[u][kb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
      const unsigned char* kp = sb + k_lane + ((ks * 4 + g4) ^ kx) * 16;
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) {
        const bf16x8_t kf = *(const bf16x8_t*)(kp + key_perm(kb, 0) * HD * 2);
#pragma unroll
        for (int u = 0; u < U; ++u)
          s[u][kb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qf[u][ks], s[u][kb], 0, 0, 0);
      }
    }
    // Blocks of context keys that are all valid need no mask (all but the last one);
    // in-block blocks and the context tail mask per element and zero V^T past kend.
    if (inblk || kb0 + kKeyBlock > kend) {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int lim1 = inblk ? e1[u] : L, lo = inblk ? lo2[u] : 0, sp = inblk ? span[u] : 0;
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int key = kb0 + key_perm(kb, 4 * g4 + r);
            const bool vis = (key < lim1) | ((unsigned)(key - lo) < (unsigned)sp);
            s[u][kb][r] = vis ? s[u][kb][r] : -INFINITY;
          }
      }
    }
    bf16x8_t pf[U][2], pfl[U][2];  // [u][t]: p = hi + lo, both bf16
#pragma unroll
    for (int u = 0; u < U; ++u) {
      float mx = -INFINITY;
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
#pragma unroll
        for (int r = 0; r < 4; ++r) mx = fmaxf(mx, s[u][kb][r]);
      mx = rows4_max(mx) * sc;                                          // block max, log2 units
      const float m_new = mx > m_run[u] + kLazyMax ? mx : m_run[u];   // reference of p
      const float m_use = m_new == -INFINITY ? 0.f : m_new;            // row sees no key yet
      float psum = 0.f;
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        uint32_t hw[4], lw[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          // slot j of k-step t holds key t*32 + g4*8 + j: kb = 2t + j/4, r = j%4
          const int kb = 2 * t + (q >> 1), r = 2 * (q & 1);
          const float p0 = __builtin_amdgcn_exp2f(fmaf(s[u][kb][r], sc, -m_use));
          const float p1 = __builtin_amdgcn_exp2f(fmaf(s[u][kb][r + 1], sc, -m_use));
          psum += p0 + p1;
          bf16x2_t h;
          h[0] = (__bf16)p0;
          h[1] = (__bf16)p1;
          hw[q] = __builtin_bit_cast(uint32_t, h);
          asm("" : "+v"(hw[q]));  // keeps the compiler from converting p0 a second time below
          bf16x2_t l;
          l[0] = (__bf16)(p0 - __uint_as_float(hw[q] << 16));
          l[1] = (__bf16)(p1 - __uint_as_float(hw[q] & 0xFFFF0000u));
          lw[q] = __builtin_bit_cast(uint32_t, l);
        }
        pf[u][t] = as_bf16x8(make_uint4(hw[0], hw[1], hw[2], hw[3]));
        pfl[u][t] = as_bf16x8(make_uint4(lw[0], lw[1], lw[2], lw[3]));
      }
      // o is rescaled only when some row of the wave moved its reference (alpha == 1 else)
      const float alpha = __builtin_amdgcn_exp2f(m_run[u] - m_use);
      l_run[u] = l_run[u] * alpha + psum;
      if (__any(m_new > m_run[u])) {
#pragma unroll
        for (int hb = 0; hb < NHB; ++hb) o[u][hb] *= alpha;
      }
      m_run[u] = m_new;
    }
    // O^T += V^T P^T over 64 keys = 2 k-steps of 32; the V^T fragment of the next product is
    // read while the current one's MFMAs run.
    const unsigned char* vp0 = sb + K_BYTES + v_lane + (g4 ^ vx) * 16;
    const unsigned char* vp1 = sb + K_BYTES + v_lane + ((4 + g4) ^ vx) * 16;
    auto vfrag = [&](int q) {
      return *(const bf16x8_t*)((q < NHB ? vp0 : vp1) + (q % NHB) * 16 * kKeyBlock * 2);
    };
    bf16x8_t vf[2];
    vf[0] = vfrag(0);
#pragma unroll
    for (int q = 0; q < 2 * NHB; ++q) {
      if (q + 1 < 2 * NHB) vf[(q + 1) & 1] = vfrag(q + 1);
      const int t = q / NHB, hb = q % NHB;
#pragma unroll
      for (int u = 0; u < U; ++u) {
        o[u][hb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf[q & 1], pf[u][t], o[u][hb], 0, 0, 0);
        o[u][hb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf[q & 1], pfl[u][t], o[u][hb], 0, 0, 0);
      }
    }
  }

#pragma unroll
  for (int u = 0; u < U; ++u) {
    const float l_tot = rows4_sum(l_run[u]);
    if (qi[u] >= nrows) continue;
    const int gi = qi[u] / a.R, row = qi[u] % a.R;
    const int h = kvh * grp + gi;
    if (a.S == 1) {
      const float inv = l_tot > 0.f ? 1.0f / l_tot : 0.f;
      bf16_t* op = (bf16_t*)a.O + (int64_t)(b * a.R + row) * (a.n_q * HD) + h * HD;
#pragma unroll
      for (int hb = 0; hb < NHB; ++hb) {
        const uint32_t w0 = f2bf(o[u][hb][0] * inv) | ((uint32_t)f2bf(o[u][hb][1] * inv) << 16);
        const uint32_t w1 = f2bf(o[u][hb][2] * inv) | ((uint32_t)f2bf(o[u][hb][3] * inv) << 16);
        *(uint2*)(op + hb * 16 + g4 * 4) = make_uint2(w0, w1);
      }
    } else {
      const int64_t base = ((int64_t)(b * a.n_q + h) * a.R + row) * a.S + split;
      if (l_tot > 0.f) {
        float* op = a.Opart + base * HD;
#pragma unroll
        for (int hb = 0; hb < NHB; ++hb)
          *(float4*)(op + hb * 16 + g4 * 4) = make_float4(o[u][hb][0], o[u][hb][1], o[u][hb][2], o[u][hb][3]);
      }
      if (g4 == 0) {
        a.MLpart[base * 2] = m_run[u];
        a.MLpart[base * 2 + 1] = l_tot;
      }
    }
  }
}

// Folds the S partials of one (request, head, row): 4 head_dim entries per thread.
// Partials with l == 0 saw no key and are skipped (their O was not written): every
// partial is loaded up front, so the loads overlap, and an unwritten one is replaced by
// zero with a select (never multiplied), so that stale memory cannot reach the result.
template <int HD>
__global__ __launch_bounds__(256) void attn_fold(AttnArgs a) {
  constexpr int TPR = HD / 4;  // threads per (request, head, row)
  constexpr int SMAX = kMaxAttnSplits;
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t task = t / TPR;
  if (task >= (int64_t)a.B * a.n_q * a.R) return;
  const int c = (int)(t % TPR);
  const int row = (int)(task % a.R);
  const int bh = (int)(task / a.R), h = bh % a.n_q, b = bh / a.n_q;
  const int64_t pbase = task * a.S;
  float2 ml[SMAX];
  float4 v[SMAX];
#pragma unroll
  for (int s = 0; s < SMAX; ++s)
    if (s < a.S) {
      ml[s] = *(const float2*)(a.MLpart + (pbase + s) * 2);
      v[s] = *(const float4*)(a.Opart + (pbase + s) * HD + c * 4);
    }
  float M = -INFINITY;
#pragma unroll
  for (int s = 0; s < SMAX; ++s)
    if (s < a.S && ml[s].y > 0.f) M = fmaxf(M, ml[s].x);
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  float Ls = 0.f;
#pragma unroll
  for (int s = 0; s < SMAX; ++s) {
    if (s >= a.S) continue;
    const bool live = ml[s].y > 0.f;
    const float w = live ? exp2f(ml[s].x - M) : 0.f;
    Ls += live ? ml[s].y * w : 0.f;
    acc.x += live ? v[s].x * w : 0.f;
    acc.y += live ? v[s].y * w : 0.f;
    acc.z += live ? v[s].z * w : 0.f;
    acc.w += live ? v[s].w * w : 0.f;
  }
  const float inv = Ls > 0.f ? 1.0f / Ls : 0.f;
  bf16_t* op = (bf16_t*)a.O + (int64_t)(b * a.R + row) * (a.n_q * HD) + h * HD + c * 4;
  const uint32_t w0 = f2bf(acc.x * inv) | ((uint32_t)f2bf(acc.y * inv) << 16);
  const uint32_t w1 = f2bf(acc.z * inv) | ((uint32_t)f2bf(acc.w * inv) << 16);
  *(uint2*)op = make_uint2(w0, w1);
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

// float32 path, second pass: one wave per (request, head, row) takes the context partial,
// then walks the row's in-block keys under the tree mask and writes the normalised O.
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
  const T* Kp = (const T*)a.Kb + (int64_t)(b * a.n_kv + kvh) * a.Rp * HD;  // [Rp][hd]
  const T* Vp = (const T*)a.Vb + (int64_t)(b * a.n_kv + kvh) * HD * a.Rp;  // [hd][Rp]
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
    for (int c = 0; c < PER; ++c) o[c] = fmaf(p, ld_f(Vp + (int64_t)(lane + 64 * c) * a.Rp + key), o[c] * al);
    M = mn;
  }
  const float inv = 1.0f / Ls;
  T* op = (T*)a.O + (int64_t)(b * a.R + row) * (a.n_q * HD) + h * HD;
#pragma unroll
  for (int c = 0; c < PER; ++c) st_f(op + lane + 64 * c, o[c] * inv);
}

template <int HD>
hipError_t run_attention_bf16(const AttnArgs& a, hipStream_t st) {
  constexpr int STAGES = kAttnStages;
  constexpr size_t lds = (size_t)STAGES * 2 * kKeyBlock * HD * 2;
  static_assert(lds <= 163840, "attention LDS ring exceeds 160 KB");
  if constexpr (lds > 65536) {
    static const hipError_t attr = hipFuncSetAttribute(
        (const void*)attn_mfma<HD, kAttnWaves, kAttnTiles, STAGES>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (attr != hipSuccess) return attr;
  }
  const int nrows = (a.n_q / a.n_kv) * a.R;
  {
    Phase ph("attn_ctx", st);
    const int grid = (nrows + kRowsPerWG - 1) / kRowsPerWG * a.S * a.B * a.n_kv;
    hipLaunchKernelGGL((attn_mfma<HD, kAttnWaves, kAttnTiles, STAGES>), dim3(grid), dim3(64 * kAttnWaves), lds, st, a);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.S == 1) return e;
  {
    Phase ph("attn_merge", st);
    const int64_t threads = (int64_t)a.B * a.n_q * a.R * (HD / 4);
    hipLaunchKernelGGL((attn_fold<HD>), dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, st, a);
  }
  return hipGetLastError();
}

template <typename T, int HD>
hipError_t run_attention_scalar(const AttnArgs& a, hipStream_t st) {
  const int waves = a.B * a.n_q * a.R;
  const int blocks = (waves + 3) / 4;
  {
    Phase ph("attn_ctx", st);
    hipLaunchKernelGGL((attn_ctx_scalar<T, HD>), dim3(blocks), dim3(256), 0, st, a);
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

int attn_rows_per_workgroup() { return kRowsPerWG; }

hipError_t launch_attention(int dtype, const AttnArgs& a, hipStream_t st) {
  if (a.Rp < a.R || a.Rp % kKeyBlock || a.S < 1 || a.S > kMaxAttnSplits) return hipErrorInvalidValue;
  if (dtype == 1) return a.hd == 128 ? run_attention_bf16<128>(a, st) : run_attention_bf16<64>(a, st);
  if (a.S != 1) return hipErrorInvalidValue;
  return a.hd == 128 ? run_attention_scalar<float, 128>(a, st) : run_attention_scalar<float, 64>(a, st);
}

}  // namespace dpara
