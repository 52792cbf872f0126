// Greedy verification, branch gather and the Markov AR head.
//
// verify: per (row, vocab chunk) a workgroup reduces its slice to one packed 64-bit
// (value, lowest index) key; one workgroup per request then reduces each row's chunk keys
// (one wave per row, one key per lane) to its argmax g_j, and one wave compares the
// drafts t_{j+1} with g_j (lane j): a ballot of the mismatches gives the accepted length
// r = index of the first mismatch (gamma if none) and the bonus g_r (Section 2.1;
// Algorithm 1, Verify).
//
// Sampling variant: the acceptance test and bonus draw of speculative sampling (Section 2.1)
// over log-sum-exp partials of the target and draft-score rows; the head steps rank
// z / T plus Gumbel noise.
//
// head: y_0 = bonus; step i computes z_i = l_i + W E(y_{i-1}) over the vocabulary in
// chunks (8 lanes per vocabulary row, E(y_{i-1}) staged in LDS) and keeps a per-chunk
// top-2; the next step's workgroups reduce those partials to y_i and the top1 - top2
// margin before starting (head equation of Section 3.2).  For ranks up to 512 (bf16) or
// 256 (float32) the step prefetches its whole weight slice (ar_step_pf); wider ranks
// walk the rows (ar_step).
#include <math.h>

#include "common.h"
#include "internal.h"

namespace dpara {
namespace {

// VEC: rows are 16-byte aligned and the chunk is read in 16-byte pieces (8 bf16 or 4 float32
// per load), several pieces in flight per thread; otherwise element by element.
template <typename T, bool VEC>
__global__ __launch_bounds__(256) void verify_partial(const T* logits, int V, int chunk, int n_chunks,
                                                      uint64_t* part) {
  __shared__ uint64_t red[4];
  const int rowid = blockIdx.y, c = blockIdx.x;
  const T* x = logits + (int64_t)rowid * V;
  const int v0 = c * chunk, v1 = min(V, v0 + chunk);
  uint64_t best = 0;
  if constexpr (VEC) {
    constexpr int EPP = 16 / sizeof(T);
#pragma unroll 4
    for (int v = v0 + threadIdx.x * EPP; v < v1; v += 256 * EPP) {
      const uint4 u = *(const uint4*)(x + v);
      const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
      for (int q = 0; q < EPP; ++q) {
        float f;
        if constexpr (sizeof(T) == 2) f = __uint_as_float(q & 1 ? (w[q >> 1] & 0xFFFF0000u) : (w[q >> 1] << 16));
        else f = __uint_as_float(w[q]);
        if (v + q < v1) {
          const uint64_t k = argmax_key(f, (uint32_t)(v + q));
          best = k > best ? k : best;
        }
      }
    }
  } else {
    for (int v = v0 + threadIdx.x; v < v1; v += 256) {
      const uint64_t k = argmax_key(ld_f(x + v), (uint32_t)v);
      best = k > best ? k : best;
    }
  }
  best = wave_max_u64(best);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = best;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint64_t m = red[0];
    for (int i = 1; i < 4; ++i) m = red[i] > m ? red[i] : m;
    part[(int64_t)rowid * n_chunks + c] = m;
  }
}

// One workgroup of 16 waves per request: wave w reduces rows w, w + 16, ... with one chunk
// partial per lane (all loads of a row in flight at once), then wave 0 compares the drafts.
constexpr int kFinWaves = 16;
__global__ __launch_bounds__(64 * kFinWaves) void verify_finalize(int gamma, int V, int n_chunks,
                                                                  const uint64_t* part, const int* spine,
                                                                  int* accept_len, int* bonus, int* target_argmax,
                                                                  int* status) {
  __shared__ int gs[64];
  const int b = blockIdx.x, wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  for (int j = wave; j <= gamma; j += kFinWaves) {
    const uint64_t* p = part + ((int64_t)b * (gamma + 1) + j) * n_chunks;
    uint64_t best = 0;
    for (int c = lane; c < n_chunks; c += 64) best = p[c] > best ? p[c] : best;
    best = wave_max_u64(best);
    if (lane == 0) gs[j] = (int)key_index(best);
  }
  __syncthreads();
  if (wave != 0) return;
  int g = 0;
  if (lane <= gamma) {
    g = gs[lane];
    if (target_argmax) target_argmax[b * (gamma + 1) + lane] = g;
  }
  bool mismatch = false;
  if (lane < gamma) {
    const int t = spine[b * (gamma + 1) + lane + 1];
    if (t < 0 || t >= V) raise_status(status, 1);
    mismatch = (t != g);
  }
  const uint64_t mask = __ballot(mismatch);
  const int r = mask ? (__ffsll((unsigned long long)mask) - 1) : gamma;
  const int bon = __shfl(g, r, kWave);
  if (lane == 0) {
    accept_len[b] = r;
    bonus[b] = bon;
  }
}


__global__ __launch_bounds__(256) void gather_branch(int gamma, int H, const float* reps, const int* accept_len,
                                                     float* G, float* G_out, bf16_t* Ghi, int64_t lo_off,
                                                     uint64_t* clear, int64_t n_clear, int* status, int* flag) {
  const int i = blockIdx.x, b = blockIdx.y;
  if (flag && i == 0 && b == 0 && threadIdx.x == 0) *flag = 0;
  for (int64_t k = ((int64_t)b * gridDim.x + i) * 256 + threadIdx.x; k < n_clear; k += (int64_t)gridDim.x * gridDim.y * 256)
    clear[k] = 0;
  int r = accept_len[b];
  if (r < 0 || r > gamma) {
    if (threadIdx.x == 0) raise_status(status, 4);
    r = r < 0 ? 0 : gamma;
  }
  const int64_t row = (int64_t)b * gamma + i;
  const float4* src = (const float4*)(reps + (((int64_t)b * (gamma + 1) + r) * gamma + i) * H);
  float4* dst = (float4*)(G + row * H);
  float4* dst2 = G_out ? (float4*)(G_out + row * H) : nullptr;
  bf16_t* hi = Ghi + row * H;
  bf16_t* lo = hi + lo_off;
  for (int k = threadIdx.x; k < H / 4; k += 256) {
    const float4 v = src[k];
    dst[k] = v;
    if (dst2) dst2[k] = v;
    const float x[4] = {v.x, v.y, v.z, v.w};
    bf16_t h[4], l[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      h[j] = f2bf(x[j]);
      l[j] = f2bf(x[j] - bf2f(h[j]));
    }
    *(uint2*)(hi + 4 * k) = make_uint2(h[0] | ((uint32_t)h[1] << 16), h[2] | ((uint32_t)h[3] << 16));
    *(uint2*)(lo + 4 * k) = make_uint2(l[0] | ((uint32_t)l[1] << 16), l[2] | ((uint32_t)l[3] << 16));
  }
}

// Rows per 8-lane group of the prefetching AR step for P 16-byte pieces per lane per row:
// NR * P <= 32 pieces (128 VGPRs) in flight per lane.
__host__ __device__ constexpr int ar_rows_per_group(int P) { return P <= 4 ? 8 : (P <= 8 ? 4 : 0); }

template <typename T>
__device__ __forceinline__ float dot_row8(const T* w, const float* e, int rank, int j);

// bf16 row: lane j of the 8-lane group loads 16-byte pieces (t*8 + j), t < rank/64.
template <>
__device__ __forceinline__ float dot_row8<bf16_t>(const bf16_t* w, const float* e, int rank, int j) {
  float acc = 0.f;
  for (int t = 0; t < rank / 64; ++t) {
    const int k0 = (t * 8 + j) * 8;
    const uint4 u = *(const uint4*)(w + k0);
    const uint32_t ws[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      acc = fmaf(__uint_as_float(ws[q] << 16), e[k0 + 2 * q], acc);
      acc = fmaf(__uint_as_float(ws[q] & 0xFFFF0000u), e[k0 + 2 * q + 1], acc);
    }
  }
  return acc;
}
template <>
__device__ __forceinline__ float dot_row8<float>(const float* w, const float* e, int rank, int j) {
  float acc = 0.f;
  for (int t = 0; t < rank / 32; ++t) {
    const int k0 = (t * 8 + j) * 4;
    const float4 u = *(const float4*)(w + k0);
    acc = fmaf(u.x, e[k0], acc);
    acc = fmaf(u.y, e[k0 + 1], acc);
    acc = fmaf(u.z, e[k0 + 2], acc);
    acc = fmaf(u.w, e[k0 + 3], acc);
  }
  return acc;
}

// Reduce the per-chunk (key1, second value) partials of one step to (y, margin).  Every
// workgroup of the next step does this redundantly (a few KB from L2) instead of a
// grid-wide handoff, so no workgroup waits on another and no device-scope fence is needed.
__device__ __forceinline__ void reduce_step(const uint64_t* pp, int n_chunks, uint64_t* rk, float* rv,
                                            int* y_out, float* m_out) {
  uint64_t K1 = 0;
  float V2 = -INFINITY;
  for (int i = threadIdx.x; i < n_chunks; i += 256) top2_merge(K1, V2, pp[2 * i], __uint_as_float((uint32_t)pp[2 * i + 1]));
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const uint64_t ok = __shfl_xor(K1, o, kWave);
    const float ov = __shfl_xor(V2, o, kWave);
    top2_merge(K1, V2, ok, ov);
  }
  const int w = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) {
    rk[w] = K1;
    rv[w] = V2;
  }
  __syncthreads();
  uint64_t k = rk[0];
  float v = rv[0];
  for (int i = 1; i < 4; ++i) top2_merge(k, v, rk[i], rv[i]);
  *y_out = (int)key_index(k);
  *m_out = key_value(k) - v;
}

// Step `step` of the AR head (1 <= step <= gamma): y_{step-1} from the previous step's
// partials (or the bonus), then this chunk's top-2 of z = l_step + W E(y_{step-1}).
// step == gamma + 1 only reduces the last step.  Partials alternate between two slots by
// step parity: part[slot][b][chunk][2].
template <typename T>
__global__ __launch_bounds__(256) void ar_step(int step, int gamma, int V, int rank, const float* logits,
                                               const T* E, const T* W, const int* bonus, int* drafts,
                                               int* next_spine, float* margins, uint64_t* part,
                                               int n_chunks, int chunk, int B, int* status, const int* only_if,
                                               Sampling smp) {
  if (only_if && *only_if == 0) return;
  __shared__ float e[1024];
  __shared__ uint64_t rk[4];
  __shared__ float rv[4];
  const int c = blockIdx.x, b = blockIdx.y;
  int y_prev;
  if (step == 1) {
    y_prev = bonus[b];
    if (y_prev < 0 || y_prev >= V) {
      if (threadIdx.x == 0 && c == 0) raise_status(status, 1);
      y_prev = 0;
    }
    if (threadIdx.x == 0 && c == 0) next_spine[b * (gamma + 1)] = y_prev;
  } else {
    const uint64_t* pp = part + ((int64_t)((step - 1) & 1) * B + b) * n_chunks * 2;
    float m;
    reduce_step(pp, n_chunks, rk, rv, &y_prev, &m);
    if (threadIdx.x == 0 && c == 0) {
      drafts[b * gamma + step - 2] = y_prev;
      next_spine[b * (gamma + 1) + step - 1] = y_prev;
      if (margins) margins[b * gamma + step - 2] = m;
    }
  }
  if (step > gamma) return;
  for (int k = threadIdx.x; k < rank; k += 256) e[k] = ld_f(E + (int64_t)y_prev * rank + k);
  __syncthreads();
  uint32_t sk0 = 0, sk1 = 0;
  if (smp.on) sampling_key(smp, sk0, sk1);
  const float* lrow = logits + ((int64_t)b * gamma + step - 1) * V;
  const int j = threadIdx.x & 7, grp = threadIdx.x >> 3;
  const int v0 = c * chunk, v1 = min(V, v0 + chunk);
  uint64_t k1 = 0;
  float v2 = -INFINITY;
  for (int v = v0 + grp; v < v1; v += 32) {
    float d = dot_row8<T>(W + (int64_t)v * rank, e, rank, j);
    d += __shfl_xor(d, 1, kWave);
    d += __shfl_xor(d, 2, kWave);
    d += __shfl_xor(d, 4, kWave);
    if (j == 0) {
      float z = lrow[v] + d;
      if (smp.on) {
        z *= smp.inv_t;
        if (smp.scores) smp.scores[((int64_t)b * gamma + step - 1) * V + v] = z;
        z += rng_gumbel(sk0, sk1, kTagHead, b, step, v);
      }
      top2_merge(k1, v2, argmax_key(z, (uint32_t)v), -INFINITY);
    }
  }
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const uint64_t ok = __shfl_xor(k1, o, kWave);
    const float ov = __shfl_xor(v2, o, kWave);
    top2_merge(k1, v2, ok, ov);
  }
  const int w = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) {
    rk[w] = k1;
    rv[w] = v2;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int i = 1; i < 4; ++i) top2_merge(rk[0], rv[0], rk[i], rv[i]);
    uint64_t* pp = part + (((int64_t)(step & 1) * B + b) * n_chunks + c) * 2;
    pp[0] = rk[0];
    pp[1] = (uint64_t)__float_as_uint(rv[0]);
  }
}

// Prefetching form of ar_step for rows of P 16-byte pieces per lane (row bytes = 128 P):
// each 8-lane group owns NR rows (grp + 32 i), and all of the workgroup's W rows and
// logits are requested before the previous step's partials are reduced, so the weight
// stream, the partial reduction and the E(y) fetch overlap instead of paying one memory
// latency per row.  Rows past V read row V-1 and are discarded.  Same arithmetic order as
// ar_step: per lane sequential over its pieces, then the 8-lane butterfly.
template <typename T, int P>
__global__ __launch_bounds__(256) void ar_step_pf(int step, int gamma, int V, int rank, const float* logits,
                                                  const T* E, const T* W, const int* bonus, int* drafts,
                                                  int* next_spine, float* margins, uint64_t* part,
                                                  int n_chunks, int chunk, int B, int* status, const int* only_if,
                                                  Sampling smp) {
  if (only_if && *only_if == 0) return;
  constexpr int NR = ar_rows_per_group(P);
  __shared__ __attribute__((aligned(16))) float e[1024];
  __shared__ uint64_t rk[4];
  __shared__ float rv[4];
  const int c = blockIdx.x, b = blockIdx.y;
  const int j = threadIdx.x & 7, grp = threadIdx.x >> 3;
  const int v0 = c * chunk;
  const size_t row_bytes = (size_t)rank * sizeof(T);

  uint4 wv[NR][P];
  float lg = -INFINITY;
  if (step <= gamma) {
#pragma unroll
    for (int i = 0; i < NR; ++i) {
      const int v = min(v0 + grp + 32 * i, V - 1);
      const unsigned char* row = (const unsigned char*)W + (size_t)v * row_bytes;
#pragma unroll
      for (int t = 0; t < P; ++t) wv[i][t] = *(const uint4*)(row + (t * 8 + j) * 16);
    }
    const int vl = v0 + grp + 32 * j;
    if (j < NR && vl < V) lg = logits[((int64_t)b * gamma + step - 1) * V + vl];
  }

  int y_prev;
  if (step == 1) {
    y_prev = bonus[b];
    if (y_prev < 0 || y_prev >= V) {
      if (threadIdx.x == 0 && c == 0) raise_status(status, 1);
      y_prev = 0;
    }
    if (threadIdx.x == 0 && c == 0) next_spine[b * (gamma + 1)] = y_prev;
  } else {
    const uint64_t* pp = part + ((int64_t)((step - 1) & 1) * B + b) * n_chunks * 2;
    float m;
    reduce_step(pp, n_chunks, rk, rv, &y_prev, &m);
    if (threadIdx.x == 0 && c == 0) {
      drafts[b * gamma + step - 2] = y_prev;
      next_spine[b * (gamma + 1) + step - 1] = y_prev;
      if (margins) margins[b * gamma + step - 2] = m;
    }
  }
  if (step > gamma) return;
  for (int k = threadIdx.x; k < rank; k += 256) e[k] = ld_f(E + (int64_t)y_prev * rank + k);
  __syncthreads();

  constexpr int EPP = 16 / sizeof(T);  // elements per 16-byte piece
  float zmine = -INFINITY;
#pragma unroll
  for (int i = 0; i < NR; ++i) {
    float d = 0.f;
#pragma unroll
    for (int t = 0; t < P; ++t) {
      const float* ek = e + (t * 8 + j) * EPP;
      const uint4 u = wv[i][t];
      const uint32_t ws[4] = {u.x, u.y, u.z, u.w};
      if constexpr (sizeof(T) == 2) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          d = fmaf(__uint_as_float(ws[q] << 16), ek[2 * q], d);
          d = fmaf(__uint_as_float(ws[q] & 0xFFFF0000u), ek[2 * q + 1], d);
        }
      } else {
#pragma unroll
        for (int q = 0; q < 4; ++q) d = fmaf(__uint_as_float(ws[q]), ek[q], d);
      }
    }
    d += __shfl_xor(d, 1, kWave);
    d += __shfl_xor(d, 2, kWave);
    d += __shfl_xor(d, 4, kWave);
    if (j == i) zmine = lg + d;
  }
  const int vmine = v0 + grp + 32 * j;
  if (smp.on && j < NR && vmine < V) {
    zmine *= smp.inv_t;
    if (smp.scores) smp.scores[((int64_t)b * gamma + step - 1) * V + vmine] = zmine;
    uint32_t sk0, sk1;
    sampling_key(smp, sk0, sk1);
    zmine += rng_gumbel(sk0, sk1, kTagHead, b, step, vmine);
  }
  uint64_t k1 = (j < NR && vmine < V) ? argmax_key(zmine, (uint32_t)vmine) : 0;
  float v2 = -INFINITY;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const uint64_t ok = __shfl_xor(k1, o, kWave);
    const float ov = __shfl_xor(v2, o, kWave);
    top2_merge(k1, v2, ok, ov);
  }
  const int w = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) {
    rk[w] = k1;
    rv[w] = v2;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int i = 1; i < 4; ++i) top2_merge(rk[0], rv[0], rk[i], rv[i]);
    uint64_t* pp = part + (((int64_t)(step & 1) * B + b) * n_chunks + c) * 2;
    pp[0] = rk[0];
    pp[1] = (uint64_t)__float_as_uint(rv[0]);
  }
}


// ------------------------------------------------------------ speculative-sampling verify
// Online (max, sum of exp(x - max)) over one row chunk; -inf sums are empty.
__device__ __forceinline__ void ms_add(float& m, float& s, float x) {
  if (x > m) {
    s = s * expf(m - x) + 1.f;
    m = x;
  } else {
    s += expf(x - m);
  }
}
__device__ __forceinline__ void ms_merge(float& m, float& s, float om, float os) {
  if (os == 0.f) return;
  if (s == 0.f) {
    m = om;
    s = os;
    return;
  }
  const float M = fmaxf(m, om);
  s = s * expf(m - M) + os * expf(om - M);
  m = M;
}

// Row r < n_trows: target row (times inv_t); otherwise draft-score row r - n_trows.  Every
// workgroup writes (max, sum) of its chunk of kLseChunk entries to part[row][chunk]; the
// 16-byte form loads all of a thread's entries into registers, takes their max, then sums
// one exponential per entry.
constexpr int kLseChunk = 4096;
template <typename T, bool VEC>
__global__ __launch_bounds__(256) void lse_partial(const T* tl, const float* sc, int V, int n_chunks, int n_trows,
                                                   float inv_t, float2* part) {
  __shared__ float rm[4], rs[4];
  const int row = blockIdx.y, c = blockIdx.x;
  const int v0 = c * kLseChunk, v1 = min(V, v0 + kLseChunk);
  float m = -INFINITY, s = 0.f;
  if (row < n_trows) {
    const T* x = tl + (int64_t)row * V;
    if constexpr (VEC) {
      constexpr int EPP = 16 / sizeof(T), NL = kLseChunk / (256 * EPP);
      float f[NL * EPP];
#pragma unroll
      for (int k = 0; k < NL; ++k) {
        const int v = v0 + (k * 256 + (int)threadIdx.x) * EPP;
        const uint4 u = v < v1 ? *(const uint4*)(x + v) : make_uint4(0, 0, 0, 0);
        const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
        for (int q = 0; q < EPP; ++q) {
          float e;
          if constexpr (sizeof(T) == 2) e = __uint_as_float(q & 1 ? (w[q >> 1] & 0xFFFF0000u) : (w[q >> 1] << 16));
          else e = __uint_as_float(w[q]);
          f[k * EPP + q] = v + q < v1 ? e * inv_t : -INFINITY;
        }
      }
      // the thread's entries are in registers: max first, then one exponential each
#pragma unroll
      for (int i = 0; i < NL * EPP; ++i) m = fmaxf(m, f[i]);
      if (m > -INFINITY) {
#pragma unroll
        for (int i = 0; i < NL * EPP; ++i) s += expf(f[i] - m);
      }
    } else {
      for (int v = v0 + threadIdx.x; v < v1; v += 256) ms_add(m, s, ld_f(x + v) * inv_t);
    }
  } else {
    const float* x = sc + (int64_t)(row - n_trows) * V;
    if constexpr (VEC) {
      constexpr int NL = kLseChunk / 1024;
      float f[NL * 4];
#pragma unroll
      for (int k = 0; k < NL; ++k) {
        const int v = v0 + (k * 256 + (int)threadIdx.x) * 4;
        const float4 q = v < v1 ? *(const float4*)(x + v) : make_float4(-INFINITY, -INFINITY, -INFINITY, -INFINITY);
        f[4 * k] = q.x;
        f[4 * k + 1] = q.y;
        f[4 * k + 2] = q.z;
        f[4 * k + 3] = q.w;
      }
#pragma unroll
      for (int i = 0; i < NL * 4; ++i) m = fmaxf(m, f[i]);
      if (m > -INFINITY) {
#pragma unroll
        for (int i = 0; i < NL * 4; ++i) s += expf(f[i] - m);
      }
    } else {
      for (int v = v0 + threadIdx.x; v < v1; v += 256) ms_add(m, s, x[v]);
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float om = __shfl_xor(m, o, kWave), os = __shfl_xor(s, o, kWave);
    ms_merge(m, s, om, os);
  }
  if ((threadIdx.x & 63) == 0) {
    rm[threadIdx.x >> 6] = m;
    rs[threadIdx.x >> 6] = s;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int i = 1; i < 4; ++i) ms_merge(m, s, rm[i], rs[i]);
    part[(int64_t)row * n_chunks + c] = make_float2(m, s);
  }
}

// One workgroup of 16 waves per request.  The waves first reduce the chunk partials of the
// request's 2 gamma + 1 rows (one partial per lane, then a shuffle merge) to log-sum-exps:
// target rows 0..gamma and draft-score rows 1..gamma.  Then wave 0, lane j (1..gamma), tests
// draft t_j against p_{j-1} (target row j-1) and q_j in log space: accepted iff
// log p - log q - log u > 0.  An out-of-range draft is flagged and never accepted.
// info[b] = (r, lse of target row r, lse of draft-score row r+1 (the residual's q), 0).
template <typename T>
__global__ __launch_bounds__(64 * kFinWaves) void spec_accept(int B, int gamma, int V, int n_chunks,
                                                              const float2* part, const T* tl, const float* sc,
                                                              const int* spine, Sampling smp, int* accept_len,
                                                              float4* info, int* status) {
  __shared__ float lse[128];  // [0, gamma]: target rows; gamma + i: draft-score row of draft i
  const int b = blockIdx.x, wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t trow0 = (int64_t)b * (gamma + 1);
  for (int j = wave; j < 2 * gamma + 1; j += kFinWaves) {
    const int64_t row = j <= gamma ? trow0 + j : (int64_t)B * (gamma + 1) + (int64_t)b * gamma + (j - gamma - 1);
    const float2* p = part + row * n_chunks;
    float m = -INFINITY, s = 0.f;
    for (int c = lane; c < n_chunks; c += 64) ms_merge(m, s, p[c].x, p[c].y);
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      const float om = __shfl_xor(m, o, kWave), os = __shfl_xor(s, o, kWave);
      ms_merge(m, s, om, os);
    }
    if (lane == 0) lse[j] = m + logf(s);
  }
  __syncthreads();
  if (wave != 0) return;
  bool reject = false;
  if (lane >= 1 && lane <= gamma) {
    const int t = spine[trow0 + lane];
    if (t < 0 || t >= V) {
      raise_status(status, 1);
      reject = true;
    } else {
      uint32_t k0, k1;
      sampling_key(smp, k0, k1);
      const float lp = ld_f(tl + (trow0 + lane - 1) * V + t) * smp.inv_t - lse[lane - 1];
      const float lq = sc[((int64_t)b * gamma + lane - 1) * V + t] - lse[gamma + lane];
      const float u = rng_uniform(k0, k1, kTagAccept, b, lane, 0);
      reject = !(lp - lq - logf(u) > 0.f);
    }
  }
  const uint64_t mask = __ballot(reject);
  const int r = mask ? (__ffsll((unsigned long long)mask) - 2) : gamma;
  if (lane == 0) {
    accept_len[b] = r;
    info[b] = make_float4((float)r, lse[r], r < gamma ? lse[gamma + r + 1] : 0.f, 0.f);
  }
}

// Bonus candidates of one chunk of kBonusChunk entries (4 per thread, loads first): keys of
// log(p - q) + G where p > q (the residual) and of log p + G (used after full acceptance, or
// should rounding leave the residual empty).
constexpr int kBonusChunk = 1024;
template <typename T>
__global__ __launch_bounds__(256) void spec_bonus_partial(int gamma, int V, int n_bchunks, const T* tl,
                                                          const float* sc, const float4* info, Sampling smp,
                                                          uint64_t* bpart) {
  constexpr int PER = kBonusChunk / 256;
  __shared__ uint64_t red[2][4];
  const int c = blockIdx.x, b = blockIdx.y;
  const float4 in = info[b];
  const int r = (int)in.x;
  const T* prow = tl + ((int64_t)b * (gamma + 1) + r) * V;
  const float* qrow = r < gamma ? sc + ((int64_t)b * gamma + r) * V : nullptr;
  float x[PER], y[PER];
#pragma unroll
  for (int k = 0; k < PER; ++k) {
    const int v = c * kBonusChunk + k * 256 + (int)threadIdx.x;
    x[k] = v < V ? ld_f(prow + v) : 0.f;
    y[k] = (qrow && v < V) ? qrow[v] : 0.f;
  }
  uint32_t k0, k1;
  sampling_key(smp, k0, k1);
  const float inv_t = smp.inv_t;
  uint64_t kres = 0, kp = 0;
#pragma unroll
  for (int k = 0; k < PER; ++k) {
    const int v = c * kBonusChunk + k * 256 + (int)threadIdx.x;
    if (v < V) {
      const float lp = x[k] * inv_t - in.y;
      const float g = rng_gumbel(k0, k1, kTagBonus, b, 0, v);
      const uint64_t a = argmax_key(lp + g, (uint32_t)v);
      kp = a > kp ? a : kp;
      if (qrow) {
        const float d = expf(lp) - expf(y[k] - in.z);
        if (d > 0.f) {
          const uint64_t kk = argmax_key(logf(d) + g, (uint32_t)v);
          kres = kk > kres ? kk : kres;
        }
      }
    }
  }
  kres = wave_max_u64(kres);
  kp = wave_max_u64(kp);
  if ((threadIdx.x & 63) == 0) {
    red[0][threadIdx.x >> 6] = kres;
    red[1][threadIdx.x >> 6] = kp;
  }
  __syncthreads();
  if (threadIdx.x < 2) {
    uint64_t m = red[threadIdx.x][0];
    for (int i = 1; i < 4; ++i) m = red[threadIdx.x][i] > m ? red[threadIdx.x][i] : m;
    bpart[((int64_t)b * n_bchunks + c) * 2 + threadIdx.x] = m;
  }
}

__global__ __launch_bounds__(64) void spec_bonus_final(int gamma, int n_bchunks, const float4* info,
                                                       const uint64_t* bpart, int* bonus) {
  const int b = blockIdx.x;
  uint64_t kres = 0, kp = 0;
  for (int c = threadIdx.x; c < n_bchunks; c += 64) {
    const uint64_t a = bpart[((int64_t)b * n_bchunks + c) * 2], p = bpart[((int64_t)b * n_bchunks + c) * 2 + 1];
    kres = a > kres ? a : kres;
    kp = p > kp ? p : kp;
  }
  kres = wave_max_u64(kres);
  kp = wave_max_u64(kp);
  if (threadIdx.x == 0) {
    const int r = (int)info[b].x;
    bonus[b] = (int)key_index((r < gamma && kres != 0) ? kres : kp);
  }
}
}  // namespace

hipError_t launch_verify(int logits_dtype, int B, int gamma, int V, const void* logits, const int* spine,
                         int* accept_len, int* bonus, int* target_argmax, uint64_t* part, int n_chunks,
                         int chunk, int* status, hipStream_t st) {
  Phase ph("verify", st);
  dim3 grid(n_chunks, B * (gamma + 1));
  const size_t esz = logits_dtype == 1 ? 2 : 4;
  const bool vec = ((uintptr_t)logits % 16 == 0) && ((size_t)V * esz % 16 == 0) && ((size_t)chunk * esz % 16 == 0);
  if (logits_dtype == 1) {
    if (vec)
      hipLaunchKernelGGL((verify_partial<bf16_t, true>), grid, dim3(256), 0, st, (const bf16_t*)logits, V, chunk,
                         n_chunks, part);
    else
      hipLaunchKernelGGL((verify_partial<bf16_t, false>), grid, dim3(256), 0, st, (const bf16_t*)logits, V, chunk,
                         n_chunks, part);
  } else {
    if (vec)
      hipLaunchKernelGGL((verify_partial<float, true>), grid, dim3(256), 0, st, (const float*)logits, V, chunk,
                         n_chunks, part);
    else
      hipLaunchKernelGGL((verify_partial<float, false>), grid, dim3(256), 0, st, (const float*)logits, V, chunk,
                         n_chunks, part);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(verify_finalize, dim3(B), dim3(64 * kFinWaves), 0, st, gamma, V, n_chunks, part, spine, accept_len,
                     bonus, target_argmax, status);
  return hipGetLastError();
}

size_t verify_sampled_bytes(int B, int gamma, int n_chunks) {
  auto up = [](size_t x) { return (x + 255) / 256 * 256; };
  const size_t n_bchunks = (size_t)n_chunks * (kLseChunk / kBonusChunk);
  return up((size_t)B * (2 * gamma + 1) * n_chunks * 8) + up((size_t)B * 16) + up((size_t)B * n_bchunks * 16);
}

hipError_t launch_verify_sampled(int logits_dtype, int B, int gamma, int V, const void* logits, const float* scores,
                                 const int* spine, const Sampling& smp, int* accept_len,
                                 int* bonus, void* scratch, int n_chunks, int chunk, int* status, hipStream_t st) {
  const float inv_t = smp.inv_t;
  if (chunk != kLseChunk || n_chunks != (V + kLseChunk - 1) / kLseChunk || gamma > 63) return hipErrorInvalidValue;
  Phase ph("verify", st);
  auto up = [](size_t x) { return (x + 255) / 256 * 256; };
  const int n_bchunks = (V + kBonusChunk - 1) / kBonusChunk;
  char* base = (char*)scratch;
  float2* part = (float2*)base;
  float4* info = (float4*)(base + up((size_t)B * (2 * gamma + 1) * n_chunks * 8));
  uint64_t* bpart = (uint64_t*)((char*)info + up((size_t)B * 16));
  const size_t esz = logits_dtype == 1 ? 2 : 4;
  const bool vec = ((uintptr_t)logits % 16 == 0) && ((uintptr_t)scores % 16 == 0) && ((size_t)V * esz % 16 == 0) &&
                   (V % 4 == 0);
  const int n_trows = B * (gamma + 1);
  dim3 g1(n_chunks, n_trows + B * gamma);
#define DPARA_LSE(TT, VV)                                                                                 \
  hipLaunchKernelGGL((lse_partial<TT, VV>), g1, dim3(256), 0, st, (const TT*)logits, scores, V, n_chunks, \
                     n_trows, inv_t, part)
  if (logits_dtype == 1) {
    if (vec) DPARA_LSE(bf16_t, true);
    else DPARA_LSE(bf16_t, false);
  } else {
    if (vec) DPARA_LSE(float, true);
    else DPARA_LSE(float, false);
  }
#undef DPARA_LSE
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const dim3 fin(64 * kFinWaves);
  if (logits_dtype == 1) {
    hipLaunchKernelGGL(spec_accept<bf16_t>, dim3(B), fin, 0, st, B, gamma, V, n_chunks, part, (const bf16_t*)logits,
                       scores, spine, smp, accept_len, info, status);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(spec_bonus_partial<bf16_t>, dim3(n_bchunks, B), dim3(256), 0, st, gamma, V, n_bchunks,
                       (const bf16_t*)logits, scores, info, smp, bpart);
  } else {
    hipLaunchKernelGGL(spec_accept<float>, dim3(B), fin, 0, st, B, gamma, V, n_chunks, part, (const float*)logits,
                       scores, spine, smp, accept_len, info, status);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(spec_bonus_partial<float>, dim3(n_bchunks, B), dim3(256), 0, st, gamma, V, n_bchunks,
                       (const float*)logits, scores, info, smp, bpart);
  }
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(spec_bonus_final, dim3(B), dim3(64), 0, st, gamma, n_bchunks, info, bpart, bonus);
  return hipGetLastError();
}

hipError_t launch_gather_branch(int B, int gamma, int H, const float* reps, const int* accept_len, float* G,
                                float* G_out, bf16_t* Ghi, uint64_t* clear, int64_t n_clear, int* status,
                                hipStream_t st, int* flag) {
  Phase ph("gather", st);
  hipLaunchKernelGGL(gather_branch, dim3(gamma, B), dim3(256), 0, st, gamma, H, reps, accept_len, G, G_out, Ghi,
                     (int64_t)B * gamma * H, clear, n_clear, status, flag);
  return hipGetLastError();
}

int ar_head_chunk(int dtype, int rank) {
  const int P = rank * (dtype == 1 ? 2 : 4) / 128;
  const int nr = ar_rows_per_group(P);
  return nr > 0 ? 32 * nr : 256;
}

template <typename T, int P>
hipError_t launch_ar_pf(dim3 grid, hipStream_t st, int step, int gamma, int V, int rank, const float* logits,
                        const void* E, const void* W, const int* bonus, int* drafts, int* next_spine,
                        float* margins, uint64_t* part, int n_chunks, int chunk, int B, int* status,
                        const int* only_if, const Sampling& smp) {
  hipLaunchKernelGGL((ar_step_pf<T, P>), grid, dim3(256), 0, st, step, gamma, V, rank, logits, (const T*)E,
                     (const T*)W, bonus, drafts, next_spine, margins, part, n_chunks, chunk, B, status, only_if,
                     smp);
  return hipGetLastError();
}

hipError_t launch_ar_head(int dtype, int B, int gamma, int V, int rank, const float* logits, const void* E,
                          const void* W, const int* bonus, int* drafts, int* next_spine, float* margins,
                          uint64_t* part, int n_chunks, int chunk, uint64_t* ppart, int ppart_grid, int* status,
                          const int* only_if, hipStream_t st, const Sampling& smp) {
  if (dtype == 1 && ppart && ppart_grid > 0) {
    const hipError_t e = launch_ar_head_persistent(B, gamma, V, rank, logits, E, W, bonus, drafts, next_spine,
                                                   margins, ppart, ppart_grid, status, only_if, st, smp);
    if (e != hipErrorNotSupported) return e;
  }
  if (chunk != ar_head_chunk(dtype, rank) || n_chunks != (V + chunk - 1) / chunk) return hipErrorInvalidValue;
  const int P = rank * (dtype == 1 ? 2 : 4) / 128;
  for (int step = 1; step <= gamma + 1; ++step) {
    Phase ph("ar_step", st);
    dim3 grid(step <= gamma ? n_chunks : 1, B);
    hipError_t e = hipErrorInvalidValue;
#define DPARA_AR_PF(TT, PP) \
  e = launch_ar_pf<TT, PP>(grid, st, step, gamma, V, rank, logits, E, W, bonus, drafts, next_spine, margins, part, \
                           n_chunks, chunk, B, status, only_if, smp)
    if (dtype == 1) {
      switch (P) {
        case 1: DPARA_AR_PF(bf16_t, 1); break;
        case 2: DPARA_AR_PF(bf16_t, 2); break;
        case 3: DPARA_AR_PF(bf16_t, 3); break;
        case 4: DPARA_AR_PF(bf16_t, 4); break;
        case 5: DPARA_AR_PF(bf16_t, 5); break;
        case 6: DPARA_AR_PF(bf16_t, 6); break;
        case 7: DPARA_AR_PF(bf16_t, 7); break;
        case 8: DPARA_AR_PF(bf16_t, 8); break;
        default:
          hipLaunchKernelGGL(ar_step<bf16_t>, grid, dim3(256), 0, st, step, gamma, V, rank, logits, (const bf16_t*)E,
                             (const bf16_t*)W, bonus, drafts, next_spine, margins, part, n_chunks, chunk, B, status,
                             only_if, smp);
          e = hipGetLastError();
      }
    } else {
      switch (P) {
        case 2: DPARA_AR_PF(float, 2); break;
        case 4: DPARA_AR_PF(float, 4); break;
        case 6: DPARA_AR_PF(float, 6); break;
        case 8: DPARA_AR_PF(float, 8); break;
        default:
          hipLaunchKernelGGL(ar_step<float>, grid, dim3(256), 0, st, step, gamma, V, rank, logits, (const float*)E,
                             (const float*)W, bonus, drafts, next_spine, margins, part, n_chunks, chunk, B, status,
                             only_if, smp);
          e = hipGetLastError();
      }
    }
#undef DPARA_AR_PF
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace dpara
