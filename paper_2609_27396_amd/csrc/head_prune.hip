// Exact bound-pruned AR head.
//
// The head step y_i = argmax_v z_v with z_v = l_v + W_v . E(y_{i-1}) (head equation of
// Section 3.2) needs the whole vocabulary only when the correction W_v . e can reorder the
// logits far down the list.  By Cauchy-Schwarz every v has
//     z_v <= l_v + max_u |W_u| |e|,
// so if K candidates C hold the K largest logits and L is the largest logit outside C,
// every v outside C has z_v <= L + max_u |W_u| |e|.  When the best and the second best z
// over C both exceed that bound, they are the top two over the whole vocabulary: the
// step's argmax and its top1 - top2 margin are exact, and the step costs K dot products of
// length ar_rank instead of a sweep over all V rows of W.
//
//   logit_topk      per (row, vocabulary split): the kTopK largest logit keys and the
//                   (kTopK+1)-th, in descending order.  The threshold is the (kTopK+1)-th
//                   largest of the 256 per-thread maxima (at least kTopK+1 elements are at
//                   or above it), found by rank counting in LDS; a second pass collects the
//                   elements at or above it and ranks them the same way.
//   w_rownorm_max   per-workgroup maxima of |W_v|^2 (16 lanes per row); the first
//                   workgroup also clears the fallback flag.
//   ar_pruned       one workgroup per request runs all gamma steps.  A 16-lane row per head
//                   row merges the split lists (one list per lane, DPP row maxima) into the
//                   global top kTopK and the bound, the (kTopK+1)-th key: every logit left
//                   out of a split's list is at most that split's last key, which no more
//                   than kTopK keys of the union exceed.  Per step, 16 lanes per candidate
//                   take the dot product W_v . e over rank slices; the candidates of a step
//                   depend on the row only, so their W and E rows are fetched three steps
//                   ahead into an LDS ring by DMA, and the winner's E row is in the ring
//                   when the step ends.
//
// A row whose candidate collection overflows, or a step whose bound does not hold, sets
// the fallback flag; the full head (launch_ar_head with only_if = flag) then recomputes
// every request and overwrites these results.  Keys are the argmax keys of common.h
// (larger value wins, the lower index on ties), as in the full head.
#include <math.h>

#include <algorithm>

#include "common.h"
#include "internal.h"

namespace dpara {
namespace {

constexpr int kTopK = 16;         // candidates kept per row
constexpr int kKeys = kTopK + 1;  // + the bound key
constexpr int kCollect = 512;     // collection buffer of the second pass
constexpr int kHiList = 64;       // hi-plane candidates rescored per branch row (off the serial path)
constexpr int kMaxGamma = 63;
constexpr int kMaxSplits = 16;
constexpr int kEmbedNormParts = 512;  // workgroups of the embedding row-norm pass
constexpr int kPrunedRing = 4;        // steps of candidate rows in flight in the pruned head

// LDS ring of the pruned head: per step, every thread's piece (RANK / 16 elements) of its
// candidate's W row and E row, moved in 16-byte (else 4-byte) DMA granules.
template <typename T, int RANK>
struct PrunedRing {
  static constexpr int kPiece = RANK / 16 * (int)sizeof(T);
  static constexpr int kGranule = kPiece % 16 == 0 ? 16 : 4;
  static constexpr int kSlot = 2 * 256 * kPiece;
  static constexpr int kListBytes = 16 * kMaxSplits * (kTopK + 1) * 8;
  static constexpr int kDynBytes = kPrunedRing * kSlot > kListBytes ? kPrunedRing * kSlot : kListBytes;
};

// EPL contiguous elements from p as float, in 16-byte (or 8-byte) pieces.
template <typename T, int EPL>
__device__ __forceinline__ void load_piece(const T* p, float (&r)[EPL]) {
  constexpr int BYTES = EPL * (int)sizeof(T);
  constexpr int PB = BYTES % 16 == 0 ? 16 : 8;
  constexpr int EPW = 4 / (int)sizeof(T);  // elements per 32-bit word
#pragma unroll
  for (int q = 0; q < BYTES / PB; ++q) {
    uint32_t w[PB / 4];
    if constexpr (PB == 16) {
      const uint4 u = ((const uint4*)p)[q];
      w[0] = u.x;
      w[1] = u.y;
      w[2] = u.z;
      w[3] = u.w;
    } else {
      const uint2 u = ((const uint2*)p)[q];
      w[0] = u.x;
      w[1] = u.y;
    }
#pragma unroll
    for (int i = 0; i < PB / 4; ++i) {
      if constexpr (EPW == 2) {
        r[(q * (PB / 4) + i) * 2] = __uint_as_float(w[i] << 16);
        r[(q * (PB / 4) + i) * 2 + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
      } else {
        r[q * (PB / 4) + i] = __uint_as_float(w[i]);
      }
    }
  }
}

__device__ __forceinline__ uint64_t row16_max_u64(uint64_t k) {
  uint64_t o = dpp_u64<kDppXor1>(k);
  k = o > k ? o : k;
  o = dpp_u64<kDppXor2>(k);
  k = o > k ? o : k;
  o = dpp_u64<kDppHalfMirror>(k);
  k = o > k ? o : k;
  o = dpp_u64<kDppMirror>(k);
  return o > k ? o : k;
}

// Rows of V float32 logits; split sp covers [sp*per, min(V, (sp+1)*per)).  With V % 4 == 0
// and per % 4 == 0 the scans read 16-byte pieces.
template <typename F>
__device__ __forceinline__ void scan_split(const float* x, int v0, int v1, bool vec, F&& fn) {
  const int tid = threadIdx.x;
  if (vec) {
    // four 16-byte loads in flight per thread
    const float4* x4 = (const float4*)x;
    const int q1 = v1 >> 2;
    for (int q = (v0 >> 2) + tid; q < q1; q += 1024) {
      float4 f[4];
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (q + 256 * u < q1) f[u] = x4[q + 256 * u];
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (q + 256 * u < q1) {
          const int v = 4 * (q + 256 * u);
          fn(f[u].x, v);
          fn(f[u].y, v + 1);
          fn(f[u].z, v + 2);
          fn(f[u].w, v + 3);
        }
    }
  } else {
    for (int v = v0 + tid; v < v1; v += 1024) {
      float f[4];
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (v + 256 * u < v1) f[u] = x[v + 256 * u];
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (v + 256 * u < v1) fn(f[u], v + 256 * u);
    }
  }
}

__global__ __launch_bounds__(256) void logit_topk(const float* logits, int V, int S, int per, uint64_t* out,
                                                  int* flag) {
  __shared__ __attribute__((aligned(16))) uint64_t tm[256];
  __shared__ uint64_t buf[kCollect];
  __shared__ uint64_t thr;
  __shared__ int cnt;
  const int row = blockIdx.y, sp = blockIdx.x, tid = threadIdx.x;
  const int v0 = sp * per, v1 = min(V, v0 + per);
  const bool vec = (V & 3) == 0 && (per & 3) == 0;
  const float* x = logits + (int64_t)row * V;

  uint64_t best = 0;
  scan_split(x, v0, v1, vec, [&](float f, int v) {
    const uint64_t k = argmax_key(f, (uint32_t)v);
    best = k > best ? k : best;
  });
  tm[tid] = best;
  if (tid == 0) {
    cnt = 0;
    thr = 0;
  }
  __syncthreads();
  // rank of this thread's maximum among the 256 (keys are unique; empty threads hold 0)
  int r = 0;
  for (int j = 0; j < 256; j += 2) {
    const uint4 u = *(const uint4*)&tm[j];
    r += (((uint64_t)u.y << 32 | u.x) > best) + (((uint64_t)u.w << 32 | u.z) > best);
  }
  if (r == kTopK && best != 0) thr = best;
  __syncthreads();
  const uint64_t T = thr;
  if (T != 0) {
    scan_split(x, v0, v1, vec, [&](float f, int v) {
      const uint64_t k = argmax_key(f, (uint32_t)v);
      if (k >= T) {
        const int pos = atomicAdd(&cnt, 1);
        if (pos < kCollect) buf[pos] = k;
      }
    });
  }
  __syncthreads();
  const int n = cnt;
  if (T == 0 || n > kCollect) {
    // not decidable here (a split of fewer than kKeys elements cannot occur: the launcher
    // keeps at least 64 per split); the full head takes over
    if (tid == 0) atomicOr(flag, 1);
    return;
  }
  uint64_t* o = out + ((int64_t)row * S + sp) * kKeys;
  for (int e = tid; e < n; e += 256) {
    const uint64_t k = buf[e];
    int rr = 0;
    for (int j = 0; j < n; ++j) rr += buf[j] > k;
    if (rr < kKeys) o[rr] = k;
  }
}

// fp32 rows -> bf16 hi + lo planes (hi = bf16(x), lo = bf16(x - hi)), one workgroup per row,
// and the planes' Euclidean norms (nrm[2 row] = |hi|, nrm[2 row + 1] = |lo|, each rounded up
// by a factor 1 + 2^-10 that covers the float32 sum of squares of up to 2^13 terms).
__global__ __launch_bounds__(256) void split_rows_norms(const float* X, int H, bf16_t* hi, bf16_t* lo, float* nrm) {
  __shared__ float red[4];
  const int64_t row = blockIdx.x;
  const float4* xr = (const float4*)(X + row * H);
  float shi = 0.f, slo = 0.f;
  for (int k = threadIdx.x; k < H / 4; k += 256) {
    const float4 v = xr[k];
    const float x[4] = {v.x, v.y, v.z, v.w};
    bf16_t h[4], l[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      h[j] = f2bf(x[j]);
      const float hf = bf2f(h[j]);
      l[j] = f2bf(x[j] - hf);
      const float lf = bf2f(l[j]);
      shi = fmaf(hf, hf, shi);
      slo = fmaf(lf, lf, slo);
    }
    *(uint2*)(hi + row * H + 4 * k) = make_uint2(h[0] | ((uint32_t)h[1] << 16), h[2] | ((uint32_t)h[3] << 16));
    *(uint2*)(lo + row * H + 4 * k) = make_uint2(l[0] | ((uint32_t)l[1] << 16), l[2] | ((uint32_t)l[3] << 16));
  }
  shi = block_sum256(shi, red);
  slo = block_sum256(slo, red);
  if (threadIdx.x == 0) {
    constexpr float up = 1.0f + 0x1p-10f;
    nrm[2 * row] = sqrtf(shi) * up;
    nrm[2 * row + 1] = sqrtf(slo) * up;
  }
}

// Per-workgroup maxima of |E_v|^2 over the rows of a [V, H] bf16 matrix (H % 8 == 0), one
// wave per row at a time.
__global__ __launch_bounds__(256) void row_norm2_max(const bf16_t* E, int V, int H, float* part) {
  __shared__ float red[4];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  float m = 0.f;
  for (int v = blockIdx.x * 4 + wave; v < V; v += gridDim.x * 4) {
    const bf16_t* er = E + (int64_t)v * H;
    float s = 0.f;
    for (int k = lane * 8; k < H; k += 512) {
      const bf16x8_t x = *(const bf16x8_t*)(er + k);
#pragma unroll
      for (int j = 0; j < 8; ++j) s = fmaf((float)x[j], (float)x[j], s);
    }
    m = fmaxf(m, wave_sum(s));
  }
  if (lane == 0) red[wave] = m;
  __syncthreads();
  if (threadIdx.x == 0) part[blockIdx.x] = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
}

// Exact logits of the candidates, from the single-plane (hi) top lists.  One wave per branch
// row: the row's kHiList hi-plane candidates are rescored with the full row and the kTopK
// largest exact logits, in descending order, plus a bound key go to the row's slots in
// `keys`.  Candidate rows of the embedding are the 16 columns of MFMA B operands (one
// 16-column block per 16 candidates) and the row's hi and lo planes fill every A row, so
// that each candidate's logit accumulates through exactly the sequence of MFMAs that the
// two-plane LM head GEMM applies to its element (per 32-deep k chunk in order: hi, then lo,
// from a zero accumulator): the rescored values are the LM head's, bit for bit.
// Bound: a v outside the hi list has l_hi_v <= L_hi (the list's own bound, slot kHiList),
// and
//   l_v <= l_hi_v + |lo . E_v| + |rounding of both sums|
//       <= L_hi + |E|max (|lo| + cacc (|hi| + |lo|)),
// with |lo . E_v| <= |lo| |E_v| (Cauchy-Schwarz) and each float32 sum of n products off by
// at most 2 n 2^-24 of the sum of their magnitudes (a bound that also holds for truncating
// adders), which Cauchy-Schwarz bounds by (|hi| + |lo|) |E_v|: cacc = 2 (2H + H) 2^-24.  A v
// in the list but not among the kTopK exact largest is at most the (kTopK+1)-th exact value.
// The bound key holds the larger of the two.
__global__ __launch_bounds__(256) void rescore_candidates(int rows, int H, int V, const bf16_t* hi, const bf16_t* lo,
                                                          const bf16_t* E, const float* nrm, const float* emax2,
                                                          float cacc, const uint64_t* hlist, uint64_t* keys) {
  static_assert(kHiList == 64 && kTopK < kHiList, "one hi-list candidate per lane");
  constexpr int NB = kHiList / 16;  // 16-column blocks
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * (blockDim.x >> 6) + wave;
  if (row >= rows) return;  // (no block-wide synchronisation below)
  const uint64_t* hr = hlist + row * (kHiList + 1);
  const int j = lane & 15, g4 = lane >> 4;
  const bf16_t* ep[NB];
#pragma unroll
  for (int c = 0; c < NB; ++c) {
    const uint64_t kc = hr[c * 16 + j];
    const uint32_t v = kc ? min(key_index(kc), (uint32_t)(V - 1)) : 0u;
    ep[c] = E + (int64_t)v * H + g4 * 8;
  }
  const bf16_t* hp = hi + row * H + g4 * 8;
  const bf16_t* lp = lo + row * H + g4 * 8;
  f32x4_t acc[NB];
#pragma unroll
  for (int c = 0; c < NB; ++c) acc[c] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  // The embedding rows are scattered over the table, so each k chunk's loads are a full
  // memory latency: chunks are loaded PD ahead in a register ring (past the end the last
  // chunk is loaded again and never used).  The MFMAs still run in k order, hi then lo.
  constexpr int PD = 4;
  const int KC = H / 32;
  bf16x8_t rh[PD], rl[PD], re[PD][NB];
  auto load = [&](int kc, bf16x8_t& h, bf16x8_t& l, bf16x8_t(&e)[NB]) {
    kc = min(kc, KC - 1);
    h = *(const bf16x8_t*)(hp + kc * 32);
    l = *(const bf16x8_t*)(lp + kc * 32);
#pragma unroll
    for (int c = 0; c < NB; ++c) e[c] = *(const bf16x8_t*)(ep[c] + kc * 32);
  };
#pragma unroll
  for (int d = 0; d < PD; ++d) load(d, rh[d], rl[d], re[d]);
  for (int kc0 = 0; kc0 < KC; kc0 += PD) {
#pragma unroll
    for (int d = 0; d < PD; ++d) {
      if (kc0 + d < KC) {
#pragma unroll
        for (int c = 0; c < NB; ++c) {
          acc[c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(rh[d], re[d][c], acc[c], 0, 0, 0);
          acc[c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(rl[d], re[d][c], acc[c], 0, 0, 0);
        }
      }
      load(kc0 + d + PD, rh[d], rl[d], re[d]);
    }
  }
  // every A row is this row, so each lane holds its column's value in every element: lane q
  // takes candidate q (block g4, column j)
  float val = acc[0][0];
#pragma unroll
  for (int c = 1; c < NB; ++c) val = g4 == c ? acc[c][0] : val;
  const uint64_t kq = hr[lane];
  const uint64_t nk = kq ? argmax_key(val, key_index(kq)) : 0;
  int rank = 0;
  for (int t = 0; t < kHiList; ++t) {
    const uint64_t o = ((uint64_t)__shfl((uint32_t)(nk >> 32), t, kWave) << 32) | __shfl((uint32_t)nk, t, kWave);
    rank += (o > nk) | ((o == nk) & (t < lane));
  }
  uint64_t* kr = keys + row * kKeys;
  if (rank < kTopK) kr[rank] = nk;
  // the (kTopK+1)-th exact value (-inf if the list holds no more keys)
  float vk = rank == kTopK && nk ? key_value(nk) : -INFINITY;
  vk = wave_max(vk);
  if (lane == 0) {
    const uint64_t kb = hr[kHiList];
    float bound = vk;
    if (kb) {
      const float e = sqrtf(*emax2) * (1.0f + 0x1p-10f);
      const float nh = nrm[2 * row], nl = nrm[2 * row + 1];
      const float delta = e * (nl + cacc * (nh + nl)) * (1.0f + 0x1p-10f);
      bound = fmaxf(bound, key_value(kb) + delta);
    }
    kr[kTopK] = argmax_key(bound, 0xFFFFFFFEu);
  }
}

// Per row: the tiles' (key1, key2, third value) triples of the top-2 GEMM epilogue ->
// the N largest keys of the row and, in slot N, a key whose value bounds every other logit
// of the row: the largest of the remaining keys and of the tiles' third values (a logit
// that is not among its tile's two largest is at most that tile's third value).  Fewer than
// N keys (a vocabulary of few tiles) leave zero keys, which never win.
template <int N>
__global__ __launch_bounds__(256) void tile_top2_merge(const uint64_t* part, int NT, uint64_t* out, int* flag) {
  static_assert(N < 256 && N < kCollect, "the threshold is a rank among 256 thread maxima");
  __shared__ __attribute__((aligned(16))) uint64_t tm[256];
  __shared__ uint64_t buf[kCollect];
  __shared__ float red[4];
  __shared__ uint64_t thr;
  __shared__ int cnt;
  const int row = blockIdx.x, tid = threadIdx.x;
  const uint64_t* pr = part + (int64_t)row * NT * 3;
  uint64_t best = 0;
  float v3 = -INFINITY;
  for (int t = tid; t < NT; t += 256) {
    const uint64_t k1 = pr[3 * t];
    best = k1 > best ? k1 : best;  // the tile's second key is smaller
    v3 = fmaxf(v3, __uint_as_float((uint32_t)pr[3 * t + 2]));
  }
  tm[tid] = best;
  v3 = wave_max(v3);
  if ((tid & 63) == 0) red[tid >> 6] = v3;
  if (tid == 0) {
    cnt = 0;
    thr = 0;
  }
  __syncthreads();
  int r = 0;
  for (int j = 0; j < 256; j += 2) {
    const uint4 u = *(const uint4*)&tm[j];
    r += (((uint64_t)u.y << 32 | u.x) > best) + (((uint64_t)u.w << 32 | u.z) > best);
  }
  if (r == N && best != 0) thr = best;
  __syncthreads();
  const uint64_t T = thr;  // 0: fewer than N + 1 threads hold a key; then every key is taken
  for (int t = tid; t < NT; t += 256)
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const uint64_t k = pr[3 * t + q];
      if (k != 0 && k >= T) {
        const int pos = atomicAdd(&cnt, 1);
        if (pos < kCollect) buf[pos] = k;
      }
    }
  __syncthreads();
  const int n = cnt;
  uint64_t* o = out + (int64_t)row * (N + 1);
  if (n > kCollect) {
    if (tid == 0) atomicOr(flag, 1);
    return;
  }
  for (int e = tid; e <= N; e += 256) o[e] = 0;
  __syncthreads();
  for (int e = tid; e < n; e += 256) {
    const uint64_t k = buf[e];
    int rr = 0;
    for (int j = 0; j < n; ++j) rr += buf[j] > k;
    if (rr <= N) o[rr] = k;
  }
  __syncthreads();
  if (tid == 0) {
    float bound = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
    if (n > N) bound = fmaxf(bound, key_value(o[N]));
    o[N] = argmax_key(bound, 0xFFFFFFFEu);
  }
}

template <typename T, int RANK>
__global__ __launch_bounds__(256) void w_rownorm_max(const T* W, int V, float* partial, int* flag) {
  constexpr int EPL = RANK / 16;
  __shared__ float red[4];
  const int tid = threadIdx.x;
  if (blockIdx.x == 0 && tid == 0) *flag = 0;
  const int per = (V + gridDim.x - 1) / gridDim.x;
  const int v0 = blockIdx.x * per, v1 = min(V, v0 + per);
  const int sub = tid & 15, grp = tid >> 4;  // a 16-lane row reads one W row
  float mx = 0.f;
  for (int v = v0 + grp; v < v1; v += 64) {  // four rows per 16-lane row in flight
    float r[4][EPL];
#pragma unroll
    for (int u = 0; u < 4; ++u)
      if (v + 16 * u < v1) load_piece<T, EPL>(W + (int64_t)(v + 16 * u) * RANK + sub * EPL, r[u]);
#pragma unroll
    for (int u = 0; u < 4; ++u)
      if (v + 16 * u < v1) {
        float s = 0.f;
#pragma unroll
        for (int j = 0; j < EPL; ++j) s = fmaf(r[u][j], r[u][j], s);
        mx = fmaxf(mx, row16_sum(s));
      }
  }
  mx = wave_max(mx);
  if ((tid & 63) == 0) red[tid >> 6] = mx;
  __syncthreads();
  if (tid == 0) partial[blockIdx.x] = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
}

// 16-byte (or 8-byte) raw pieces of EPT elements, converted to float at use.
template <typename T, int EPT>
struct RawPiece {
  static constexpr int WORDS = EPT * (int)sizeof(T) / 4;
  uint32_t w[WORDS];
  __device__ __forceinline__ void load(const T* p) {
    if constexpr (WORDS % 4 == 0) {
#pragma unroll
      for (int q = 0; q < WORDS / 4; ++q) {
        const uint4 u = ((const uint4*)p)[q];
        w[4 * q] = u.x;
        w[4 * q + 1] = u.y;
        w[4 * q + 2] = u.z;
        w[4 * q + 3] = u.w;
      }
    } else {
#pragma unroll
      for (int q = 0; q < WORDS / 2; ++q) {
        const uint2 u = ((const uint2*)p)[q];
        w[2 * q] = u.x;
        w[2 * q + 1] = u.y;
      }
    }
  }
  // The piece a DMA ring slot holds for `lane`: chunk q of GR bytes at base + (q * 64 + lane) * GR.
  // 16-byte chunks are read by inline ds_read_b128 with the LDS wait in the same block: for
  // ordinary loads of a DMA-filled buffer the compiler waits for every outstanding DMA first,
  // which would drain the ring each step.
  template <int GR>
  __device__ __forceinline__ void load_lds(const unsigned char* base, int lane) {
    if constexpr (GR == 16) {
      static_assert(WORDS == 4 || WORDS == 8 || WORDS == 16, "1, 2 or 4 chunks");
      uint4 u[WORDS / 4];
      const uint32_t a = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) unsigned char*)base + lane * 16;
      if constexpr (WORDS == 4) {
        asm volatile("ds_read_b128 %0, %1\n\ts_waitcnt lgkmcnt(0)" : "=v"(u[0]) : "v"(a) : "memory");
      } else if constexpr (WORDS == 8) {
        asm volatile("ds_read_b128 %0, %2\n\tds_read_b128 %1, %2 offset:1024\n\ts_waitcnt lgkmcnt(0)"
                     : "=v"(u[0]), "=v"(u[1]) : "v"(a) : "memory");
      } else {
        asm volatile(
            "ds_read_b128 %0, %4\n\tds_read_b128 %1, %4 offset:1024\n\tds_read_b128 %2, %4 offset:2048\n\t"
            "ds_read_b128 %3, %4 offset:3072\n\ts_waitcnt lgkmcnt(0)"
            : "=v"(u[0]), "=v"(u[1]), "=v"(u[2]), "=v"(u[3]) : "v"(a) : "memory");
      }
#pragma unroll
      for (int q = 0; q < WORDS / 4; ++q) {
        w[4 * q] = u[q].x;
        w[4 * q + 1] = u[q].y;
        w[4 * q + 2] = u[q].z;
        w[4 * q + 3] = u[q].w;
      }
    } else {
#pragma unroll
      for (int q = 0; q < WORDS * 4 / GR; ++q) w[q] = *(const uint32_t*)(base + (q * 64 + lane) * 4);
    }
  }
  __device__ __forceinline__ float at(int j) const {
    if constexpr (sizeof(T) == 2) return __uint_as_float((j & 1) ? (w[j >> 1] & 0xFFFF0000u) : (w[j >> 1] << 16));
    else return __uint_as_float(w[j]);
  }
};

// One direct global->LDS DMA instruction of GR bytes a lane (lane l's bytes land at l * GR
// past the wave-uniform LDS address).
template <int GR>
__device__ __forceinline__ void dma_granule(const void* g, void* l) {
  if constexpr (GR == 16) __builtin_amdgcn_global_load_lds(g, (lds_void_t*)l, 16, 0, 0);
  else __builtin_amdgcn_global_load_lds(g, (lds_void_t*)l, 4, 0, 0);
}

// Workgroup barrier for LDS traffic only: the wave's LDS accesses complete, then s_barrier.
// (__syncthreads also waits for every outstanding global load, which would drain the
// candidate-row ring each step.)
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

template <typename T, int RANK>
__global__ __launch_bounds__(256) void ar_pruned(int gamma, int V, int S, const uint64_t* cand,
                                                 const float* wpart, int n_wpart, const T* E, const T* W,
                                                 const int* bonus, int* drafts, int* next_spine, float* margins,
                                                 int* flag, int* status, const int* accept_len,
                                                 const int* pre_flag, float inv_t) {
  constexpr int EPT = RANK / 16;
  constexpr int D = kPrunedRing;
  constexpr int PB = PrunedRing<T, RANK>::kPiece, GR = PrunedRing<T, RANK>::kGranule;
  constexpr int NQ = PB / GR;                          // DMA instructions per piece
  constexpr int SLOT = PrunedRing<T, RANK>::kSlot;     // W pieces, then E pieces, of every thread
  __shared__ uint64_t ck[kMaxGamma][kKeys];            // per row: top kTopK keys, then the bound key
  __shared__ float es[RANK];                           // E(y_{i-1})
  __shared__ float zs[kTopK];
  __shared__ float ms[kMaxGamma];
  __shared__ int ys[kMaxGamma];
  __shared__ float red[4];
  __shared__ int ybc, stop;
  // dynamic LDS: the split lists of 16 head rows during the merge, then the candidate-row ring
  extern __shared__ __attribute__((aligned(16))) unsigned char dyn[];
  auto lists = (uint64_t(*)[kMaxSplits * kKeys])dyn;
  const int b = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int kc = tid >> 4, slice = tid & 15;  // 16-lane row kc: candidate kc, rank slice `slice`

  int y0 = bonus[b];
  if (y0 < 0 || y0 >= V) {
    if (tid == 0) raise_status(status, 1);
    y0 = 0;
  }
  if (tid == 0) {
    next_spine[b * (gamma + 1)] = y0;
    // some candidate row was not decidable: the full head recomputes everything
    const int pre = pre_flag ? *pre_flag : 0;
    if (pre && b == 0) atomicOr(flag, 1);
    stop = *flag | pre;
  }
  // candidate rows of this request: its gamma head rows, or (precomputed candidates of every
  // branch) the rows of its accepted branch
  int row0 = b * gamma;
  if (accept_len) row0 = (b * (gamma + 1) + min(max(accept_len[b], 0), gamma)) * gamma;
  float wm = 0.f;
  for (int i = tid; i < n_wpart; i += 256) wm = fmaxf(wm, wpart[i]);
  wm = wave_max(wm);
  if (lane == 0) red[wave] = wm;
  if (tid < RANK) es[tid] = ld_f(E + (int64_t)y0 * RANK + tid);

  // merge: 16 head rows at a time, lane `slice` of row kc walks split list `slice`
  for (int j0 = 0; j0 < gamma; j0 += 16) {
    const int nrow = min(16, gamma - j0);
    // the 16 rows' lists are contiguous in cand: every load of a thread is issued before the
    // first store to LDS (one memory round trip instead of one per element)
    constexpr int kPer = (16 * kMaxSplits * kKeys + 255) / 256;
    const int n = nrow * S * kKeys;
    const uint64_t* src = cand + (int64_t)(row0 + j0) * S * kKeys;
    uint64_t t[kPer];
#pragma unroll
    for (int u = 0; u < kPer; ++u) t[u] = tid + 256 * u < n ? src[tid + 256 * u] : 0;
#pragma unroll
    for (int u = 0; u < kPer; ++u)
      if (tid + 256 * u < n) {
        const int i = tid + 256 * u;
        lists[i / (S * kKeys)][i % (S * kKeys)] = t[u];
      }
    __syncthreads();
    if (kc < nrow) {
      int pos = 0;
      uint64_t head = slice < S ? lists[kc][slice * kKeys] : 0;
      for (int t = 0; t < kKeys; ++t) {
        const uint64_t m = row16_max_u64(head);
        if (slice == 0) ck[j0 + kc][t] = m;
        if (head == m && head != 0) {
          ++pos;
          head = pos < kKeys ? lists[kc][slice * kKeys + pos] : 0;
        }
      }
    }
    __syncthreads();
  }
  if (stop) return;
  const float wmax = sqrtf(fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]))) * (1.0f + 1e-5f);
  // the sampled head ranks l / T + G + (W_v . e) / T: the correction and its bound scale by 1/T
  // (exactly 1 for the greedy head)
  const float wmax_t = wmax * inv_t;

  // Step s's (1-based) candidate rows go to ring slot s % D by direct global->LDS DMA: each
  // thread's W piece (and E piece) of its candidate row, chunk q of every lane of a wave in
  // one instruction (lane l's GR bytes land at the wave's base + l * GR).  A thread reads back
  // only the bytes its own lane fetched, so a wave needs only its own vmcnt wait, and D - 1
  // steps stay in flight.  Steps past gamma reload step gamma's rows (in bounds, never used);
  // candidate indices are clamped into the vocabulary (keys of a complete list always are).
  // The loop issues no other vector-memory access: the drafts are kept in LDS and written
  // after it, and every exit drains the ring first.
  auto fetch = [&](int s) {
    const int v = (int)min(key_index(ck[min(s, gamma) - 1][kc]), (uint32_t)(V - 1));
    const unsigned char* gw = (const unsigned char*)(W + (int64_t)v * RANK + slice * EPT);
    const unsigned char* ge = (const unsigned char*)(E + (int64_t)v * RANK + slice * EPT);
    unsigned char* sl = dyn + (s % D) * SLOT + wave * 64 * PB;
#pragma unroll
    for (int q = 0; q < NQ; ++q) dma_granule<GR>(gw + q * GR, sl + q * 64 * GR);
#pragma unroll
    for (int q = 0; q < NQ; ++q) dma_granule<GR>(ge + q * GR, sl + 256 * PB + q * 64 * GR);
  };
  __syncthreads();  // the merge's reads of the lists are done before the ring overwrites them
#pragma unroll
  for (int s = 1; s < D; ++s) fetch(s);

  for (int i = 1; i <= gamma; ++i) {
    fetch(i + D - 1);
    wait_vmcnt<(D - 1) * 2 * NQ>();  // step i's pieces have landed
    __builtin_amdgcn_sched_barrier(0);
    const unsigned char* sl = dyn + (i % D) * SLOT + wave * 64 * PB;
    RawPiece<T, EPT> wp;
    wp.template load_lds<GR>(sl, lane);
    float d = 0.f, ee = 0.f;
#pragma unroll
    for (int j = 0; j < EPT; ++j) {
      const float ej = es[slice * EPT + j];
      d = fmaf(wp.at(j), ej, d);
      ee = fmaf(ej, ej, ee);
    }
    d = row16_sum(d);
    ee = row16_sum(ee);
    const uint64_t key = ck[i - 1][kc];
    if (slice == 0) zs[kc] = key ? key_value(key) + d * inv_t : -INFINITY;  // fewer than kTopK candidates
    lds_barrier();
    if (tid < 16) {  // the top two of z over the 16 candidates, one lane each
      uint64_t k1 = argmax_key(zs[tid], key_index(ck[i - 1][tid]));
      float v2 = -INFINITY;
      top2_merge(k1, v2, dpp_u64<kDppXor1>(k1), dpp_f<kDppXor1>(v2));
      top2_merge(k1, v2, dpp_u64<kDppXor2>(k1), dpp_f<kDppXor2>(v2));
      top2_merge(k1, v2, dpp_u64<kDppHalfMirror>(k1), dpp_f<kDppHalfMirror>(v2));
      top2_merge(k1, v2, dpp_u64<kDppMirror>(k1), dpp_f<kDppMirror>(v2));
      if (tid == 0) {
        const float lb = key_value(ck[i - 1][kTopK]);
        const float bound = lb + wmax_t * sqrtf(ee) + 1e-4f + 1e-5f * fabsf(lb);
        const bool ok = v2 > bound;
        const int y = (int)key_index(k1);
        ys[i - 1] = y;
        ms[i - 1] = key_value(k1) - v2;
        stop = ok ? 0 : 1;
        ybc = y;
      }
    }
    lds_barrier();
    if (stop) {
      wait_vmcnt<0>();
      if (tid == 0) atomicOr(flag, 2);
      return;
    }
    if ((int)key_index(key) == ybc) {  // the winner's row holds E(y_i)
      RawPiece<T, EPT> ep;
      ep.template load_lds<GR>(sl + 256 * PB, lane);
#pragma unroll
      for (int j = 0; j < EPT; ++j) es[slice * EPT + j] = ep.at(j);
    }
    lds_barrier();
  }
  wait_vmcnt<0>();  // the D - 1 fetches past the last step
  for (int i = tid; i < gamma; i += 256) {
    drafts[b * gamma + i] = ys[i];
    next_spine[b * (gamma + 1) + i + 1] = ys[i];
    if (margins) margins[b * gamma + i] = ms[i];
  }
}

// Perturbed head logits of the sampling variant: P[row][v] = l[row][v] * inv_t + G, with G
// the Gumbel noise of head step i = row % gamma + 1 of request row / gamma (the same draw the
// full sampled head adds).
__global__ __launch_bounds__(256) void perturb_logits(int gamma, int V, const float* L, float* P, Sampling smp) {
  const int row = blockIdx.y, b = row / gamma, i = row % gamma + 1;
  uint32_t k0, k1;
  sampling_key(smp, k0, k1);
  const int64_t o = (int64_t)row * V;
  for (int v = blockIdx.x * 256 + threadIdx.x; v < V; v += gridDim.x * 256)
    P[o + v] = L[o + v] * smp.inv_t + rng_gumbel(k0, k1, kTagHead, b, i, v);
}

// Draft scores once the drafts are known, as a GEMM: the previous tokens' E rows
// (row b * gamma + i - 1 holds E(y_{i-1}), y_0 the bonus) times W^T, then
// s = (l + c) * inv_t.  The gather also turns the pruned head's fallback flag into `ok`
// (1 when every step was proven: the full head, when it runs, writes the scores itself); c
// goes to scratch and only the finishing pass, which checks ok, writes the scores.
template <typename T>
__global__ __launch_bounds__(256) void gather_prev_e(int gamma, int V, int rank, const T* E, const int* bonus,
                                                     const int* drafts, T* rows, const int* flag, int* ok) {
  const int row = blockIdx.x, b = row / gamma, i = row % gamma;  // row's step i + 1 reads y_i
  if (row == 0 && threadIdx.x == 0) *ok = (*flag == 0) ? 1 : 0;
  int y = i == 0 ? bonus[b] : drafts[b * gamma + i - 1];
  y = min(max(y, 0), V - 1);
  for (int k = threadIdx.x; k < rank; k += 256) rows[(int64_t)row * rank + k] = E[(int64_t)y * rank + k];
}

__global__ __launch_bounds__(256) void max_of(const float* parts, int n, float* out) {
  __shared__ float red[4];
  float m = 0.f;
  for (int i = threadIdx.x; i < n; i += 256) m = fmaxf(m, parts[i]);
  m = wave_max(m);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = m;
  __syncthreads();
  if (threadIdx.x == 0) *out = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
}

__global__ __launch_bounds__(256) void finish_scores(int64_t n, const float* L, const float* C, float* S, float inv_t,
                                                     const int* ok) {
  if (*ok == 0) return;
  for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < n; e += (int64_t)gridDim.x * 256) {
    const float z = L[e] + C[e];
    S[e] = z * inv_t;
  }
}

}  // namespace

template <typename T, int RANK>
hipError_t launch_pruned(int B, int gamma, int V, int S, const uint64_t* cand, const float* wpart, int nw,
                         const void* E, const void* W, const int* bonus, int* drafts, int* next_spine,
                         float* margins, int* flag, int* status, const int* accept_len, const int* pre_flag,
                         float inv_t, hipStream_t st) {
  constexpr int lds = PrunedRing<T, RANK>::kDynBytes;
  static_assert(lds + 16384 <= 163840, "pruned-head LDS exceeds 160 KB");
  auto kern = ar_pruned<T, RANK>;
  static const hipError_t attr = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, lds);
  if (attr != hipSuccess) return attr;
  hipLaunchKernelGGL(kern, dim3(B), dim3(256), lds, st, gamma, V, S, cand, wpart, nw, (const T*)E,
                     (const T*)W, bonus, drafts, next_spine, margins, flag, status, accept_len, pre_flag, inv_t);
  return hipGetLastError();
}

hipError_t launch_wnorm(int dtype, int rank, const void* W, int V, float* wpart, int* flag, hipStream_t st) {
  const int nw = 512;
#define DPARA_WNORM(TT, RK) \
  hipLaunchKernelGGL((w_rownorm_max<TT, RK>), dim3(nw), dim3(256), 0, st, (const TT*)W, V, wpart, flag)
  if (dtype == 1) {
    if (rank == 64) DPARA_WNORM(bf16_t, 64);
    else if (rank == 128) DPARA_WNORM(bf16_t, 128);
    else DPARA_WNORM(bf16_t, 256);
  } else {
    if (rank == 64) DPARA_WNORM(float, 64);
    else if (rank == 128) DPARA_WNORM(float, 128);
    else DPARA_WNORM(float, 256);
  }
#undef DPARA_WNORM
  return hipGetLastError();
}

hipError_t dispatch_pruned(int dtype, int rank, int B, int gamma, int V, int S, const uint64_t* cand,
                           const float* wpart, int nw, const void* E, const void* W, const int* bonus, int* drafts,
                           int* next_spine, float* margins, int* flag, int* status, const int* accept_len,
                           const int* pre_flag, float inv_t, hipStream_t st) {
#define DPARA_PRUNED(TT, RK)                                                                                   \
  return launch_pruned<TT, RK>(B, gamma, V, S, cand, wpart, nw, E, W, bonus, drafts, next_spine, margins, flag, \
                               status, accept_len, pre_flag, inv_t, st)
  if (dtype == 1) {
    if (rank == 64) DPARA_PRUNED(bf16_t, 64);
    if (rank == 128) DPARA_PRUNED(bf16_t, 128);
    DPARA_PRUNED(bf16_t, 256);
  }
  if (rank == 64) DPARA_PRUNED(float, 64);
  if (rank == 128) DPARA_PRUNED(float, 128);
  DPARA_PRUNED(float, 256);
#undef DPARA_PRUNED
}

int head_prune_splits(int rows, int V) {
  int S = 256 / (rows > 0 ? rows : 1);
  if (S > kMaxSplits) S = kMaxSplits;
  while (S > 1 && V / S < 64) --S;
  return S < 1 ? 1 : S;
}

int head_prune_wparts() { return 512; }

size_t head_cand_bytes(int B, int gamma) { return 4096 + (size_t)B * (gamma + 1) * gamma * kKeys * 8; }
size_t head_cand_part_bytes(int B, int gamma, int V) { return (size_t)B * (gamma + 1) * gamma * ((V + 127) / 128) * 24; }

size_t head_row_cand_bytes(int rows) { return 4096 + (size_t)rows * kKeys * 8; }

// Candidates (kTopK exact logits and a bound key) of `rows` float32 rows against the bf16
// embedding: split into hi/lo planes, hi-plane top-2 GEMM, merge into kHiList keys a row,
// exact rescoring.  With wnorm_pre the |W_v|^2 pass is skipped (the caller passes the
// prepared maximum to the steps) and only the overflow flag is cleared.
static hipError_t launch_row_candidates(int rows, int H, int V, int rank, const float* reps, const void* embed,
                                 const void* W, const float* emax2_pre, const float* wnorm_pre, void* cand,
                                 bf16_t* split, uint64_t* part, void* scratch, hipStream_t st) {
  int* overflow = (int*)cand;
  float* wpart = (float*)((unsigned char*)cand + 256);
  uint64_t* keys = (uint64_t*)((unsigned char*)cand + 4096);
  const int NT = (V + 127) / 128;
  bf16_t* hi = split;
  bf16_t* lo = split + (int64_t)rows * H;
  // scratch: the hi lists (kHiList + 1 keys a row), then |hi|, |lo| a row, then the
  // embedding norm partials and their maximum
  uint64_t* hlist = (uint64_t*)scratch;
  float* nrm = (float*)(hlist + (int64_t)rows * (kHiList + 1));
  float* eparts = nrm + 2 * (int64_t)rows;
  Phase ph("lm_head", st);
  hipLaunchKernelGGL(split_rows_norms, dim3(rows), dim3(256), 0, st, reps, H, hi, lo, nrm);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if ((e = wnorm_pre ? launch_clear_status(overflow, st) : launch_wnorm(1, rank, W, V, wpart, overflow, st)) !=
      hipSuccess)
    return e;  // (the |W_v|^2 pass also clears `overflow`)
  const float* emax2 = emax2_pre;
  if (!emax2) {  // one pass over the embedding
    hipLaunchKernelGGL(row_norm2_max, dim3(kEmbedNormParts), dim3(256), 0, st, (const bf16_t*)embed, V, H, eparts);
    hipLaunchKernelGGL(max_of, dim3(1), dim3(256), 0, st, eparts, kEmbedNormParts, eparts + kEmbedNormParts);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    emax2 = eparts + kEmbedNormParts;
  }
  // top lists from the hi plane alone: half the work of the two-plane product
  GemmArgs g{};
  g.A = hi;
  g.lda = H;
  g.B0 = g.B1 = g.B2 = embed;
  g.n1 = g.n2 = V;
  g.M = rows;
  g.N = V;
  g.K = H;
  g.C = part;
  g.ldc = NT;
  if ((e = launch_gemm(A_BF16, EPI_TOP2, g, st)) != hipSuccess) return e;
  hipLaunchKernelGGL(tile_top2_merge<kHiList>, dim3(rows), dim3(256), 0, st, part, NT, hlist, overflow);
  const float cacc = (float)(6.0 * H / 16777216.0);
  // one wave a workgroup: at batch 1 (272 rows) the rows spread over all CUs (636 -> 606 us for
  // the whole candidates pass against four rows a workgroup)
  hipLaunchKernelGGL(rescore_candidates, dim3(rows), dim3(64), 0, st, rows, H, V, hi, lo,
                     (const bf16_t*)embed, nrm, emax2, cacc, hlist, keys);
  return hipGetLastError();
}

hipError_t launch_branch_candidates(int B, int gamma, int H, int V, int rank, const float* reps, const void* embed,
                                    const void* W, const float* emax2_pre, void* cand, bf16_t* split, uint64_t* part,
                                    void* scratch, hipStream_t st) {
  if (!head_prune_supported(1, gamma, V, rank) || B < 1 || H % 64) return hipErrorNotSupported;
  return launch_row_candidates(B * (gamma + 1) * gamma, H, V, rank, reps, embed, W, emax2_pre, nullptr, cand, split,
                               part, scratch, st);
}

hipError_t launch_head_ranked(int B, int gamma, int H, int V, int rank, const float* G, const void* embed,
                              const void* E, const void* W, const float* emax2_pre, const float* wnorm_pre,
                              const int* bonus, int* drafts, int* next_spine, float* margins, int* flag, int* status,
                              void* cand, bf16_t* split, uint64_t* part, void* scratch, hipStream_t st) {
  if (!head_prune_supported(1, gamma, V, rank) || B < 1 || H % 64) return hipErrorNotSupported;
  hipError_t e = launch_row_candidates(B * gamma, H, V, rank, G, embed, W, emax2_pre, wnorm_pre, cand, split, part,
                                       scratch, st);
  if (e != hipSuccess) return e;
  const int* overflow = (const int*)cand;
  const float* wpart = wnorm_pre ? wnorm_pre : (const float*)((const unsigned char*)cand + 256);
  const uint64_t* keys = (const uint64_t*)((const unsigned char*)cand + 4096);
  Phase ph("ar_step", st);
  if ((e = launch_clear_status(flag, st)) != hipSuccess) return e;
  return dispatch_pruned(1, rank, B, gamma, V, 1, keys, wpart, wnorm_pre ? 1 : head_prune_wparts(), E, W, bonus,
                         drafts, next_spine, margins, flag, status, nullptr, overflow, 1.0f, st);
}

size_t head_cand_scratch_bytes(int B, int gamma) {
  const size_t rows = (size_t)B * (gamma + 1) * gamma;
  return rows * (kHiList + 1) * 8 + (rows * 2 + kEmbedNormParts + 1) * 4;
}

hipError_t launch_embed_prepare(const void* embed, int V, int H, float* parts, float* out, hipStream_t st) {
  if (H % 8) return hipErrorNotSupported;
  hipLaunchKernelGGL(row_norm2_max, dim3(kEmbedNormParts), dim3(256), 0, st, (const bf16_t*)embed, V, H, parts);
  hipLaunchKernelGGL(max_of, dim3(1), dim3(256), 0, st, parts, kEmbedNormParts, out);
  return hipGetLastError();
}

hipError_t launch_head_from_candidates(int B, int gamma, int V, int rank, const void* cand, const void* E,
                                       const void* W, const int* accept_len, const int* bonus, int* drafts,
                                       int* next_spine, float* margins, int* flag, int* status, hipStream_t st) {
  if (!head_prune_supported(1, gamma, V, rank) || B < 1) return hipErrorNotSupported;
  const int* overflow = (const int*)cand;
  const float* wpart = (const float*)((const unsigned char*)cand + 256);
  const uint64_t* keys = (const uint64_t*)((const unsigned char*)cand + 4096);
  Phase ph("ar_step", st);
  hipError_t e = launch_clear_status(flag, st);
  if (e != hipSuccess) return e;
  return dispatch_pruned(1, rank, B, gamma, V, 1, keys, wpart, head_prune_wparts(), E, W, bonus, drafts, next_spine,
                         margins, flag, status, accept_len, overflow, 1.0f, st);
}

bool head_prune_supported(int dtype, int gamma, int V, int rank) {
  return gamma >= 1 && gamma <= kMaxGamma && V >= 64 && (rank == 64 || rank == 128 || rank == 256) &&
         (dtype == 0 || dtype == 1);
}

size_t head_prune_cand_bytes(int rows, int V) { return (size_t)rows * head_prune_splits(rows, V) * kKeys * 8; }

hipError_t launch_head_pruned(int dtype, int B, int gamma, int V, int rank, const float* logits, const void* E,
                              const void* W, const int* bonus, int* drafts, int* next_spine, float* margins,
                              uint64_t* cand, float* wpart, int* flag, int* status, hipStream_t st, float inv_t,
                              const float* wnorm_pre, bool flag_cleared) {
  if (!head_prune_supported(dtype, gamma, V, rank) || B < 1) return hipErrorNotSupported;
  const int rows = B * gamma;
  const int S = head_prune_splits(rows, V);
  const int per = ((V + S - 1) / S + 3) / 4 * 4;
  int nw = head_prune_wparts();
  Phase ph("ar_step", st);
  // the weights' max row norm: prepared once (one float), or one pass over W here (which also
  // clears the fallback flag)
  hipError_t e = wnorm_pre ? (flag_cleared ? hipSuccess : launch_clear_status(flag, st))
                           : launch_wnorm(dtype, rank, W, V, wpart, flag, st);
  if (e != hipSuccess) return e;
  if (wnorm_pre) {
    wpart = const_cast<float*>(wnorm_pre);
    nw = 1;
  }
  hipLaunchKernelGGL(logit_topk, dim3(S, rows), dim3(256), 0, st, logits, V, S, per, cand, flag);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  return dispatch_pruned(dtype, rank, B, gamma, V, S, cand, wpart, nw, E, W, bonus, drafts, next_spine, margins, flag,
                         status, nullptr, nullptr, inv_t, st);
}

hipError_t launch_perturb_logits(int B, int gamma, int V, const float* logits, float* P, const Sampling& smp,
                                 hipStream_t st) {
  const int gx = min((V + 255) / 256, 64);
  hipLaunchKernelGGL(perturb_logits, dim3(gx, B * gamma), dim3(256), 0, st, gamma, V, logits, P, smp);
  return hipGetLastError();
}

hipError_t launch_draft_scores(int dtype, int B, int gamma, int V, int rank, const float* logits, const void* E,
                               const void* W, const int* bonus, const int* drafts, const Sampling& smp,
                               const int* flag, void* rows, float* cbuf, int* ok, hipStream_t st) {
  const int R = B * gamma;
  if (dtype == 1)
    hipLaunchKernelGGL(gather_prev_e<bf16_t>, dim3(R), dim3(256), 0, st, gamma, V, rank, (const bf16_t*)E, bonus,
                       drafts, (bf16_t*)rows, flag, ok);
  else
    hipLaunchKernelGGL(gather_prev_e<float>, dim3(R), dim3(256), 0, st, gamma, V, rank, (const float*)E, bonus,
                       drafts, (float*)rows, flag, ok);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  GemmArgs g{};
  g.A = rows;
  g.lda = rank;
  g.B0 = g.B1 = g.B2 = W;
  g.n1 = g.n2 = V;
  g.M = R;
  g.N = V;
  g.K = rank;
  g.C = cbuf;
  g.ldc = V;
  g.only_if = ok;  // (kernels that ignore it only waste work: the finishing pass checks ok)
  if ((e = launch_gemm(dtype == 1 ? A_BF16 : A_F32, EPI_STORE_F32, g, st)) != hipSuccess) return e;
  const int64_t n = (int64_t)R * V;
  const int grid = (int)std::min<int64_t>((n + 255) / 256, 4096);
  hipLaunchKernelGGL(finish_scores, dim3(grid), dim3(256), 0, st, n, logits, cbuf, smp.scores, smp.inv_t, ok);
  return hipGetLastError();
}

hipError_t launch_head_prepare(int dtype, int rank, const void* W, int V, float* parts, int* scratch_flag, float* out,
                               hipStream_t st) {
  hipError_t e = launch_wnorm(dtype, rank, W, V, parts, scratch_flag, st);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(max_of, dim3(1), dim3(256), 0, st, parts, head_prune_wparts(), out);
  return hipGetLastError();
}

}  // namespace dpara
