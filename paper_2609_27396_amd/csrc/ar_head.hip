// Persistent AR head (head equation of Section 3.2, Algorithm 1's head loop) for bf16
// drafters: one launch runs all gamma serial steps.  The sampling variant draws
// y_i ~ softmax(z_i / T) by ranking z_i / T plus Gumbel noise from the counter-based
// generator (request, step and vocabulary index in the counter) instead of z_i.
//
// Each step computes z_i = l_i + W E(y_{i-1}) over the vocabulary and y_i = argmax z_i.
// Reading the V x r matrix W from HBM at every step dominates the per-step kernels; here
// every workgroup keeps its slice of W in registers for the whole launch, so W is read
// once.  Workgroup = NW waves; wave w owns 16*NRB vocabulary rows as MFMA B-operand
// fragments (640 rows per workgroup).  Per step the workgroup stages E(y_{i-1}) of every request in LDS
// (A operand, up to 16 requests) and one v_mfma_f32_16x16x32_bf16 chain per 16-row block
// gives W E for all requests at once.
//
// Steps are chained by a grid-wide exchange without fences: each workgroup publishes, per
// request, its partial top-2 as two 64-bit words (key with the step tag in its low bits;
// second value with the tag) using device-coherent (agent-scope) relaxed atomic stores,
// and every workgroup polls all partials with device-coherent loads until every tag shows
// the step.  Each word carries its own tag, so no ordering between words is assumed.
// Partials alternate between two slots by step parity; a workgroup can only reach step
// i+2 after every workgroup has published step i+1, i.e. finished reading step i.  The
// tags are cleared (kernel boundary) before each launch.  Polls are bounded: a workgroup
// that waits longer than the spin limit raises the status bit and returns, so the grid
// always drains.  The grid must be co-resident (one workgroup per CU); the launcher
// checks occupancy and otherwise reports hipErrorNotSupported so the caller falls back
// to the per-step kernels.
#include <math.h>

#include "common.h"
#include "internal.h"

namespace dpara {
namespace {

constexpr int kArpMaxB = 16;         // requests per launch (the MFMA's 16 rows)
constexpr int kArpTagBits = 14;      // step tag in the low bits of the key word
constexpr uint32_t kArpIdxMask = 0x3FFFFu;  // vocabulary index field: V <= 2^18
constexpr int kArpMaxGrid = 256;     // polling covers up to 16 partials per thread at 16 requests
constexpr int kArpStatusTimeout = 16;

// Key word: high 32 bits = order-preserving value bits, then (index complement, 18 bits),
// then the tag.  Larger key = larger value, ties to the lower index.
__device__ __forceinline__ uint64_t arp_key(float v, uint32_t idx) {
  uint32_t u = __float_as_uint(v);
  u = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return ((uint64_t)u << 32) | ((uint64_t)(kArpIdxMask - idx) << kArpTagBits);
}
__device__ __forceinline__ uint32_t arp_index(uint64_t k) {
  return kArpIdxMask - (uint32_t)((k & 0xFFFFFFFFu) >> kArpTagBits);
}
__device__ __forceinline__ float arp_value(uint64_t k) {
  uint32_t u = (uint32_t)(k >> 32);
  u = (u & 0x80000000u) ? (u & 0x7FFFFFFFu) : ~u;
  return __uint_as_float(u);
}
// (key1, second value) merge; keys carry no tag here.
__device__ __forceinline__ void arp_merge(uint64_t& k1, float& v2, uint64_t ok1, float ov2) {
  const float va = k1 ? arp_value(k1) : -INFINITY;
  const float vb = ok1 ? arp_value(ok1) : -INFINITY;
  if (ok1 > k1) {
    v2 = fmaxf(fmaxf(v2, ov2), va);
    k1 = ok1;
  } else {
    v2 = fmaxf(fmaxf(v2, ov2), vb);
  }
}

__device__ __forceinline__ void store_dev(uint64_t* p, uint64_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t load_dev(const uint64_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// part: [2 slots][kArpMaxB][G][2] uint64 (key word, value word).
// Reduces step `s` (tags == s) for every request into ys/ms (LDS).  Returns false on timeout.
// The workgroup's threads are split evenly over the requests (tpr = 256 / bpad threads per
// request, bpad = B rounded up to a power of two), each reading ceil(G / tpr) partials in
// batches of 4, so a small batch polls all partials in one memory round trip.
__device__ bool arp_poll(const uint64_t* part, int s, int B, int G, int V, uint32_t spin_limit, int* ys, float* ms,
                         uint64_t* rkw, float* rvw) {
  int bpad = 1;
  while (bpad < B) bpad <<= 1;
  const int tpr = (int)blockDim.x / bpad;
  const int t = threadIdx.x, b = t / tpr, j = t % tpr;
  const int per = (G + tpr - 1) / tpr;
  const uint64_t* slot = part + ((int64_t)(s & 1) * kArpMaxB + b) * G * 2;
  const uint32_t tag = (uint32_t)s & ((1u << kArpTagBits) - 1);
  uint64_t K1 = 0;
  float V2 = -INFINITY;
  for (int q0 = 0; q0 < per; q0 += 4) {  // uniform
    uint32_t it = 0;
    while (true) {
      bool ok = true;
      uint64_t kw[4], vw[4];
      if (b < B) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int i = min(j + tpr * (q0 + q), G - 1);
          vw[q] = load_dev(slot + 2 * i + 1);
          kw[q] = load_dev(slot + 2 * i);
        }
#pragma unroll
        for (int q = 0; q < 4; ++q)
          if (j + tpr * (q0 + q) < G)
            ok = ok && ((uint32_t)kw[q] & ((1u << kArpTagBits) - 1)) == tag && (uint32_t)vw[q] == (uint32_t)s;
      }
      if (__syncthreads_and(ok)) {
        if (b < B) {
#pragma unroll
          for (int q = 0; q < 4; ++q)
            if (j + tpr * (q0 + q) < G)
              arp_merge(K1, V2, kw[q] & ~(uint64_t)((1u << kArpTagBits) - 1), __uint_as_float((uint32_t)(vw[q] >> 32)));
        }
        break;
      }
      if (++it > spin_limit) return false;
      __builtin_amdgcn_s_sleep(1);
    }
  }
  const int span = tpr < 64 ? tpr : 64;  // lanes of one request within a wave
  for (int o = 1; o < span; o <<= 1) {
    const uint64_t ok1 = __shfl_xor(K1, o, kWave);
    const float ov = __shfl_xor(V2, o, kWave);
    arp_merge(K1, V2, ok1, ov);
  }
  if (tpr > 64) {  // a request spans several waves: combine their results
    const int wave = t >> 6;
    if ((t & 63) == 0) {
      rkw[wave] = K1;
      rvw[wave] = V2;
    }
    __syncthreads();
    if (j == 0 && b < B) {
      for (int w = 1; w < tpr / 64; ++w) arp_merge(K1, V2, rkw[wave + w], rvw[wave + w]);
    }
  }
  if (b < B && j == 0) {
    ys[b] = min((int)arp_index(K1), V - 1);  // K1 is a real row key unless every z was NaN
    ms[b] = arp_value(K1) - V2;
  }
  return true;
}

// Branch-free top-2 tracking: (k1, v1) best key and its value, v2 second-best value.
struct Top2 {
  uint64_t k1;
  float v1, v2;
};
__device__ __forceinline__ void top2_add(Top2& t, uint64_t k, float z) {
  const bool better = k > t.k1;
  t.v2 = fmaxf(t.v2, better ? t.v1 : z);
  t.v1 = better ? z : t.v1;
  t.k1 = better ? k : t.k1;
}
__device__ __forceinline__ void top2_join(Top2& t, const Top2& o) {
  const bool better = o.k1 > t.k1;
  t.v2 = fmaxf(fmaxf(t.v2, o.v2), better ? t.v1 : o.v1);
  t.v1 = better ? o.v1 : t.v1;
  t.k1 = better ? o.k1 : t.k1;
}

// SAMPLE: the sampling variant ranks s + Gumbel noise, s = z * inv_t (and stores s when asked).
template <int NKB, int NRB, int NW, bool SAMPLE>
__global__ __launch_bounds__(64 * NW) void ar_head_persistent(int gamma, int V, int B, const float* logits,
                                                                     const bf16_t* E, const bf16_t* W,
                                                                     const int* bonus, int* drafts,
                                                                     int* next_spine, float* margins,
                                                                     uint64_t* part, int* status,
                                                                     uint32_t spin_limit, const int* only_if,
                                                                     Sampling smp) {
  // Every workgroup reads the same flag, so all of them leave together.
  if (only_if && *only_if == 0) return;
  constexpr int RANK = NKB * 32;
  constexpr int ROWS_WAVE = 16 * NRB;
  constexpr int ROWS_WG = NW * ROWS_WAVE;
  constexpr int LCH = ROWS_WG / 4;  // 16-byte logit chunks per request
  constexpr int ESTRIDE = RANK + 8;  // bf16 per staged E row (padding spreads LDS banks)
  static_assert((kArpMaxB * LCH) % (64 * NW) == 0, "logit staging must split into whole DMA rounds");
  __shared__ __attribute__((aligned(16))) bf16_t es[kArpMaxB * ESTRIDE];
  __shared__ __attribute__((aligned(16))) float lgs[kArpMaxB * ROWS_WG];  // this step's logits of the slice
  __shared__ float gs[SAMPLE ? kArpMaxB * ROWS_WG : 1];                    // this step's Gumbel noise of the slice
  __shared__ int ys[kArpMaxB];
  __shared__ float ms[kArpMaxB];
  __shared__ uint64_t rk[NW][kArpMaxB];
  __shared__ float rv[NW][kArpMaxB];
  __shared__ int bail;
  const int G = gridDim.x, wg = blockIdx.x;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, lr = lane & 15, lg = lane >> 4;
  const int vbase = (wg * NW + wave) * ROWS_WAVE;

  // W fragments: lane (lr, lg) holds W[vbase + rb*16 + lr][kb*32 + lg*8 .. +8].  Rows past
  // V read row V-1; their results are never used.
  bf16x8_t wf[NRB][NKB];
#pragma unroll
  for (int rb = 0; rb < NRB; ++rb) {
    const int v = min(vbase + rb * 16 + lr, V - 1);
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb) wf[rb][kb] = *(const bf16x8_t*)(W + (int64_t)v * RANK + kb * 32 + lg * 8);
  }
  if (tid < kArpMaxB) {
    int y = 0;
    if (tid < B) {
      y = bonus[tid];
      if (y < 0 || y >= V) {
        if (wg == 0) raise_status(status, 1);
        y = 0;
      }
      if (wg == 0) next_spine[tid * (gamma + 1)] = y;
    }
    ys[tid] = y;
  }

  const int v0 = wg * ROWS_WG;
  uint32_t sk0 = 0, sk1 = 0;
  if constexpr (SAMPLE) sampling_key(smp, sk0, sk1);
  for (int s = 1; s <= gamma; ++s) {
    // this step's logits of the slice -> LDS by DMA (independent of y): LDS chunk c holds
    // request c / LCH, rows v0 + 4*(c % LCH) .. +3 (chunks past V re-read the last full
    // chunk of the row and are never used)
    for (int c0 = 0; c0 < B * LCH; c0 += 64 * NW) {
      const int c = c0 + wave * 64 + lane;
      const int b = min(c / LCH, B - 1);
      const int v = min(v0 + 4 * (c % LCH), V - 4);
      __builtin_amdgcn_global_load_lds((const void*)(logits + ((int64_t)b * gamma + s - 1) * V + v),
                                       (lds_void_t*)(lgs + 4 * (c0 + wave * 64)), 16, 0, 0);
    }
    if constexpr (SAMPLE) {
      // the noise does not depend on y: drawn here, it overlaps the wait for the partials
#pragma unroll 1
      for (int e = tid; e < B * ROWS_WG; e += 64 * NW) {
        const int v = v0 + e % ROWS_WG;
        gs[e] = v < V ? rng_gumbel(sk0, sk1, kTagHead, e / ROWS_WG, s, v) : 0.f;
      }
    }
    if (s > 1) {
      const bool okp = arp_poll(part, s - 1, B, G, V, spin_limit, ys, ms, &rk[0][0], &rv[0][0]);
      if (tid == 0) bail = !okp;
      __syncthreads();
      if (bail) {
        if (tid == 0) raise_status(status, kArpStatusTimeout);
        return;
      }
      if (wg == 0 && tid < B) {
        drafts[tid * gamma + s - 2] = ys[tid];
        next_spine[tid * (gamma + 1) + s - 1] = ys[tid];
        if (margins) margins[tid * gamma + s - 2] = ms[tid];
      }
    } else {
      __syncthreads();
    }
    // stage E(y) rows (16-byte pieces); rows of absent requests are zero
    for (int c = tid; c < kArpMaxB * (RANK / 8); c += 64 * NW) {
      const int b = c / (RANK / 8), k = (c % (RANK / 8)) * 8;
      uint4 u = make_uint4(0, 0, 0, 0);
      if (b < B) u = *(const uint4*)(E + (int64_t)ys[b] * RANK + k);
      *(uint4*)&es[b * ESTRIDE + k] = u;
    }
    __builtin_amdgcn_s_waitcnt(0);  // this wave's logit DMA has landed
    __syncthreads();

    // z = l + E W^T: C[request 4*lg + i][row lr] of each 16-row block.  Only the first
    // min(B, 4) requests of each lane group can exist (uniform loop bound).
    const int IMAX = B < 4 ? B : 4;
    Top2 t2[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) t2[i] = Top2{0, -INFINITY, -INFINITY};
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb) {
      f32x4_t acc = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb) {
        const bf16x8_t ea = *(const bf16x8_t*)&es[lr * ESTRIDE + kb * 32 + lg * 8];
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ea, wf[rb][kb], acc, 0, 0, 0);
      }
      const int v = vbase + rb * 16 + lr;
      const int vl = wave * ROWS_WAVE + rb * 16 + lr;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        if (i >= IMAX) break;
        const int b = 4 * lg + i;
        const bool valid = v < V && b < B;
        float z = lgs[min(b, B - 1) * ROWS_WG + vl] + acc[i];
        if constexpr (SAMPLE) {
          if (valid) {
            z *= smp.inv_t;
            lgs[b * ROWS_WG + vl] = z;  // read once above: now the score, copied out below
            z += gs[b * ROWS_WG + vl];
          }
        }
        top2_add(t2[i], valid ? arp_key(z, (uint32_t)v) : 0ull, valid ? z : -INFINITY);
      }
    }
    // reduce over the 16 rows of the lane group, then over the waves
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      if (i >= IMAX) break;
#pragma unroll
      for (int o = 1; o < 16; o <<= 1) {
        Top2 ot;
        ot.k1 = __shfl_xor(t2[i].k1, o, kWave);
        ot.v1 = __shfl_xor(t2[i].v1, o, kWave);
        ot.v2 = __shfl_xor(t2[i].v2, o, kWave);
        top2_join(t2[i], ot);
      }
      if (lr == 0) {
        rk[wave][4 * lg + i] = t2[i].k1;
        rv[wave][4 * lg + i] = t2[i].v2;
      }
    }
    __syncthreads();
    if (tid < B) {
      uint64_t K = rk[0][tid];
      float V2 = rv[0][tid];
      for (int w = 1; w < NW; ++w) arp_merge(K, V2, rk[w][tid], rv[w][tid]);
      uint64_t* e = part + (((int64_t)(s & 1) * kArpMaxB + tid) * G + wg) * 2;
      store_dev(e + 1, ((uint64_t)__float_as_uint(V2) << 32) | (uint32_t)s);
      store_dev(e, K | ((uint32_t)s & ((1u << kArpTagBits) - 1)));
    }
    if constexpr (SAMPLE) {
      if (smp.scores) {  // the slice's scores z / T, row by row (the barrier above ordered them)
        for (int e = tid; e < B * ROWS_WG; e += 64 * NW) {
          const int v = v0 + e % ROWS_WG;
          if (v < V) smp.scores[((int64_t)(e / ROWS_WG) * gamma + s - 1) * V + v] = lgs[e];
        }
        __syncthreads();  // before the next step's logit DMA overwrites lgs
      }
    }
  }
  // y_gamma: only workgroup 0 needs it
  if (wg != 0) return;
  const bool okp = arp_poll(part, gamma, B, G, V, spin_limit, ys, ms, &rk[0][0], &rv[0][0]);
  if (!okp) {
    if (tid == 0) raise_status(status, kArpStatusTimeout);
    return;
  }
  __syncthreads();
  if (tid < B) {
    drafts[tid * gamma + gamma - 1] = ys[tid];
    next_spine[tid * (gamma + 1) + gamma] = ys[tid];
    if (margins) margins[tid * gamma + gamma - 1] = ms[tid];
  }
}

template <int NKB, int NRB, int NW, bool SAMPLE>
hipError_t arp_launch(int B, int gamma, int V, const float* logits, const void* E, const void* W, const int* bonus,
                      int* drafts, int* next_spine, float* margins, uint64_t* part, int part_grid, int* status,
                      const int* only_if, hipStream_t st, const Sampling& smp) {
  constexpr int ROWS_WG = NW * 16 * NRB;
  const int G = (V + ROWS_WG - 1) / ROWS_WG;
  if (G > part_grid || G > kArpMaxGrid) return hipErrorNotSupported;
  int dev = 0, cus = 0, per_cu = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e == hipSuccess)
    e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, ar_head_persistent<NKB, NRB, NW, SAMPLE>, 64 * NW, 0);
  if (e != hipSuccess) return e;
  if (G > per_cu * cus) return hipErrorNotSupported;  // not co-resident: the caller falls back
  const uint32_t spin_limit = 1u << 17;  // polls of ~2 us: ~0.3 s before a workgroup gives up
  Phase ph("ar_step", st);
  hipLaunchKernelGGL((ar_head_persistent<NKB, NRB, NW, SAMPLE>), dim3(G), dim3(64 * NW), 0, st, gamma, V, B, logits,
                     (const bf16_t*)E, (const bf16_t*)W, bonus, drafts, next_spine, margins, part, status,
                     spin_limit, only_if, smp);
  return hipGetLastError();
}

}  // namespace

// 8 waves x 5 16-row blocks (up to 160 registers of W per lane at rank 256, two waves per
// SIMD): a workgroup covers 640 vocabulary rows.  Wider ranks do not fit one workgroup per
// CU and use the step kernels.
int ar_persistent_grid(int rank, int V) {
  if (rank != 64 && rank != 128 && rank != 256) return 0;
  const int rows = 640;
  return (V + rows - 1) / rows;
}

hipError_t launch_ar_head_persistent(int B, int gamma, int V, int rank, const float* logits, const void* E,
                                     const void* W, const int* bonus, int* drafts, int* next_spine, float* margins,
                                     uint64_t* part, int part_grid, int* status, const int* only_if, hipStream_t st,
                                     const Sampling& smp) {
  if (B < 1 || B > kArpMaxB || V > (int)kArpIdxMask + 1 || V % 4 || V < 4 || gamma < 1 ||
      gamma >= (1 << kArpTagBits) || (uintptr_t)logits % 16)
    return hipErrorNotSupported;
#define DPARA_ARP(NKB)                                                                                         \
  (smp.on ? arp_launch<NKB, 5, 8, true>(B, gamma, V, logits, E, W, bonus, drafts, next_spine, margins, part,     \
                                        part_grid, status, only_if, st, smp)                                     \
          : arp_launch<NKB, 5, 8, false>(B, gamma, V, logits, E, W, bonus, drafts, next_spine, margins, part,    \
                                         part_grid, status, only_if, st, smp))
  switch (rank) {
    case 64: return DPARA_ARP(2);
    case 128: return DPARA_ARP(4);
    case 256: return DPARA_ARP(8);
    default: return hipErrorNotSupported;
  }
#undef DPARA_ARP
}

}  // namespace dpara
