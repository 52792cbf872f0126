// Device-side helpers shared by the DPara HIP kernels (gfx950, wave64).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dpara {

typedef uint16_t bf16_t;  // bfloat16 storage (upper half of an IEEE float32)
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;

__device__ __forceinline__ float bf2f(bf16_t h) { return __uint_as_float(((uint32_t)h) << 16); }

// float32 -> bfloat16, round to nearest, ties to even (finite inputs).
__device__ __forceinline__ bf16_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (bf16_t)(u >> 16);
}

template <typename T> __device__ __forceinline__ float ld_f(const T* p);
template <> __device__ __forceinline__ float ld_f<float>(const float* p) { return *p; }
template <> __device__ __forceinline__ float ld_f<bf16_t>(const bf16_t* p) { return bf2f(*p); }

template <typename T> __device__ __forceinline__ void st_f(T* p, float v);
template <> __device__ __forceinline__ void st_f<float>(float* p, float v) { *p = v; }
template <> __device__ __forceinline__ void st_f<bf16_t>(bf16_t* p, float v) { *p = f2bf(v); }

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
  return v;
}

// Block-wide sum for any block of NW waves.  `red` must hold NW floats.
template <int NW>
__device__ __forceinline__ float block_sum(float v, float* red) {
  v = wave_sum(v);
  const int w = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  float t = 0.f;
#pragma unroll
  for (int i = 0; i < NW; ++i) t += red[i];
  return t;
}

// Block-wide sum for blockDim.x == 256 (4 waves).  `red` must hold 4 floats.
__device__ __forceinline__ float block_sum256(float v, float* red) {
  v = wave_sum(v);
  const int w = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  return red[0] + red[1] + red[2] + red[3];
}

// Generic LDS pointer type of the direct global->LDS DMA builtin.
typedef __attribute__((address_space(3))) void lds_void_t;

// Row layout of one request (Section 3.2): rows 0..gamma are the spine t_0..t_gamma;
// row gamma+1 + r*gamma + (i-1) is mask i of branch r.  Position offset from the
// context length: spine j -> j; branch r mask i -> r + i.
__device__ __forceinline__ int row_pos_offset(int row, int gamma) {
  if (row <= gamma) return row;
  const int k = row - gamma - 1;
  return k / gamma + k % gamma + 1;
}

// Debug builds (DPARA_DEBUG_LDS_POISON=1) fill a kernel's LDS ring with NaN bit patterns
// before its first DMA, so that a fragment read of any LDS byte the DMA did not write turns
// the outputs into NaN, which the parity tests catch.  The fill completes (waitcnt + barrier)
// before the first DMA is issued.  A no-op otherwise.
#ifndef DPARA_DEBUG_LDS_POISON
#define DPARA_DEBUG_LDS_POISON 0
#endif
template <int BYTES>
__device__ __forceinline__ void debug_poison_lds(unsigned char* smem) {
  if constexpr (DPARA_DEBUG_LDS_POISON != 0) {
    static_assert(BYTES % 16 == 0, "the ring is a whole number of 16-byte chunks");
    for (int i = threadIdx.x; i < BYTES / 16; i += blockDim.x)
      ((uint4*)smem)[i] = make_uint4(0xFFFFFFFFu, 0xFFFFFFFFu, 0xFFFFFFFFu, 0xFFFFFFFFu);
    __syncthreads();
  }
}

// Wait until at most N vector-memory loads (DMA included) of this wave are outstanding.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  // gfx9 s_waitcnt encoding: vmcnt[3:0] | expcnt[6:4] | lgkmcnt[11:8] | vmcnt_hi[15:14];
  // expcnt and lgkmcnt are left at their maxima (no wait on them).
  __builtin_amdgcn_s_waitcnt((N & 0xF) | (0x7 << 4) | (0xF << 8) | (((N >> 4) & 3) << 14));
}

// Cross-lane moves inside 16-lane rows by DPP (no LDS round trip): quad_perm xor 1 and
// xor 2, then the half-row and row mirrors.  After the four steps every lane of a row
// holds the row's reduction.
template <int CTRL>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, 0xF, 0xF, false);
}
constexpr int kDppXor1 = 0xB1, kDppXor2 = 0x4E, kDppHalfMirror = 0x141, kDppMirror = 0x140;
template <int CTRL>
__device__ __forceinline__ float dpp_f(float v) { return __uint_as_float(dpp_u32<CTRL>(__float_as_uint(v))); }
template <int CTRL>
__device__ __forceinline__ uint64_t dpp_u64(uint64_t v) {
  return ((uint64_t)dpp_u32<CTRL>((uint32_t)(v >> 32)) << 32) | dpp_u32<CTRL>((uint32_t)v);
}
__device__ __forceinline__ float row16_sum(float v) {
  v += dpp_f<kDppXor1>(v);
  v += dpp_f<kDppXor2>(v);
  v += dpp_f<kDppHalfMirror>(v);
  v += dpp_f<kDppMirror>(v);
  return v;
}
__device__ __forceinline__ float row16_max(float v) {
  v = fmaxf(v, dpp_f<kDppXor1>(v));
  v = fmaxf(v, dpp_f<kDppXor2>(v));
  v = fmaxf(v, dpp_f<kDppHalfMirror>(v));
  v = fmaxf(v, dpp_f<kDppMirror>(v));
  return v;
}

// Orderable 64-bit key: larger value wins, and on equal values the LOWER index wins.
__device__ __forceinline__ uint64_t argmax_key(float v, uint32_t idx) {
  uint32_t u = __float_as_uint(v);
  u = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return ((uint64_t)u << 32) | (uint64_t)(0xFFFFFFFFu - idx);
}
__device__ __forceinline__ uint32_t key_index(uint64_t k) { return 0xFFFFFFFFu - (uint32_t)(k & 0xFFFFFFFFu); }
__device__ __forceinline__ float key_value(uint64_t k) {
  uint32_t u = (uint32_t)(k >> 32);
  u = (u & 0x80000000u) ? (u & 0x7FFFFFFFu) : ~u;
  return __uint_as_float(u);
}
__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    uint64_t w = __shfl_xor(v, o, kWave);
    v = w > v ? w : v;
  }
  return v;
}

// Merge (key1, second-best value) pairs.
__device__ __forceinline__ void top2_merge(uint64_t& k1, float& v2, uint64_t ok1, float ov2) {
  const float va = k1 ? key_value(k1) : -INFINITY;
  const float vb = ok1 ? key_value(ok1) : -INFINITY;
  if (ok1 > k1) {
    v2 = fmaxf(fmaxf(v2, ov2), va);
    k1 = ok1;
  } else {
    v2 = fmaxf(fmaxf(v2, ov2), vb);
  }
}

// The two largest argmax keys of a set and the third largest value (-inf if none).
struct Top3 {
  uint64_t k1 = 0, k2 = 0;
  float v3 = -INFINITY;
  __device__ __forceinline__ static float val(uint64_t k) { return k ? key_value(k) : -INFINITY; }
  __device__ __forceinline__ void add(uint64_t k) {
    if (k > k1) {
      v3 = fmaxf(v3, val(k2));
      k2 = k1;
      k1 = k;
    } else if (k > k2) {
      v3 = fmaxf(v3, val(k2));
      k2 = k;
    } else {
      v3 = fmaxf(v3, val(k));
    }
  }
  __device__ __forceinline__ static Top3 merge(const Top3& a, const Top3& b) {
    Top3 m = a;
    m.v3 = fmaxf(a.v3, b.v3);
    m.add(b.k1);
    m.add(b.k2);
    return m;
  }
  template <int CTRL>
  __device__ __forceinline__ Top3 shifted() const {
    Top3 o;
    o.k1 = dpp_u64<CTRL>(k1);
    o.k2 = dpp_u64<CTRL>(k2);
    o.v3 = dpp_f<CTRL>(v3);
    return o;
  }
  // merge over the 16 lanes of a DPP row: every lane ends with the row's result
  __device__ __forceinline__ Top3 row16() const {
    Top3 m = *this;
    m = merge(m, m.shifted<kDppXor1>());
    m = merge(m, m.shifted<kDppXor2>());
    m = merge(m, m.shifted<kDppHalfMirror>());
    m = merge(m, m.shifted<kDppMirror>());
    return m;
  }
};

// Status word (int32 at byte offset 0 of the workspace).
__device__ __forceinline__ void raise_status(int* status, int bit) { atomicOr(status, bit); }

// Counter-based random numbers for the sampling variant: word 0 of Philox4x32-10 (Salmon,
// Moraes, Dror and Shaw, SC 2011) of counter (c0, c1, c2, c3) under key (k0, k1).  Each round
// multiplies words 0 and 2 by the two Philox multipliers, xors the high halves into words 1
// and 3 with the round key, and the key advances by the two Weyl constants.
__device__ __forceinline__ uint32_t philox_word0(uint32_t k0, uint32_t k1, uint32_t c0, uint32_t c1, uint32_t c2,
                                                 uint32_t c3) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    const uint32_t h0 = __umulhi(0xD2511F53u, c0), l0 = 0xD2511F53u * c0;
    const uint32_t h2 = __umulhi(0xCD9E8D57u, c2), l2 = 0xCD9E8D57u * c2;
    c0 = h2 ^ c1 ^ k0;
    c1 = l2;
    c2 = h0 ^ c3 ^ k1;
    c3 = l0;
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
  return c0;
}
// Random-number purposes (counter word 3).
constexpr uint32_t kTagHead = 1, kTagAccept = 2, kTagBonus = 3;
// Uniform in (0, 1) from the top 23 bits k of a word: (2k + 1) / 2^24, exact in float32.
__device__ __forceinline__ float u01_of(uint32_t w) { return (float)((w >> 9) * 2u + 1u) * 0x1p-24f; }
// U(key; tag, request b, position i, index v) and its Gumbel transform -log(-log u).
__device__ __forceinline__ float rng_uniform(uint32_t k0, uint32_t k1, uint32_t tag, int b, int i, int v) {
  return u01_of(philox_word0(k0, k1, (uint32_t)v, (uint32_t)i, (uint32_t)b, tag));
}
__device__ __forceinline__ float rng_gumbel(uint32_t k0, uint32_t k1, uint32_t tag, int b, int i, int v) {
  return -logf(-logf(rng_uniform(k0, k1, tag, b, i, v)));
}

// RoPE angle for position `pos`, rotation pair p of head_dim hd, in float64 so that large
// positions keep full float32 accuracy in cos/sin.
__device__ __forceinline__ void rope_cs(int pos, int p, int hd, double base, float* c, float* s) {
  const double inv = pow(base, -2.0 * (double)p / (double)hd);
  const double a = (double)pos * inv;
  double sd, cd;
  sincos(a, &sd, &cd);
  *c = (float)cd;
  *s = (float)sd;
}

}  // namespace dpara
