// Dense projections of the drafter: C[M, N] (op)= A[M, K] . B[N, K]^T.
//
// bf16 path: v_mfma_f32_16x16x32_bf16 kernels with fp32 accumulation and fused
// epilogues (store fp32 or split-K fp32 planes, SwiGLU -> bf16, per-tile top-2 keys).
// gemm_pipe_kernel streams both operands through a multi-stage direct-to-LDS ring; the LM
// head's fp32 A operand arrives as two bf16 planes (hi + lo) that both meet every weight
// tile.  gemm_adir_kernel (M <= 320) takes A in MFMA fragment order straight into registers
// and only the weights through LDS.  Tile orders are XCD-aware: the tiles that share one
// weight tile run on the same XCD back to back, so a weight tile is fetched from HBM once
// and served to the others from that XCD's L2.
// float32 path: a plain LDS-tiled FMA kernel for the float32 model configuration.
#include "common.h"
#include "internal.h"

namespace dpara {
namespace {


// silu(g) = g / (1 + e^-g) from the hardware exp2 and reciprocal (about 1 ulp each, far below
// the bf16 rounding of the result; e^-g -> inf for very negative g gives g * 0 = -0).
__device__ __forceinline__ float silu_f(float g) {
  return g * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(g * -1.4426950408889634f));
}

// Logical tile for physical workgroup p: tiles are split into 8 contiguous ranges, one per
// XCD (workgroups are dispatched round-robin over the 8 XCDs), M fastest inside a range (or
// inside a group of 8 M tiles, below).
__device__ __forceinline__ void tile_of(int p, int MT, int NT, int& mt, int& nt) {
  const int total = MT * NT;
  const int per = total >> 3;
  int L = p;
  if (p < (per << 3)) L = (p & 7) * per + (p >> 3);
  // At 16 or more M tiles, groups of 8 M tiles, M fastest inside a group: the 32 workgroups
  // an XCD runs at once then cover about 8 M x 4 N tiles (each A tile read by 4, each weight
  // tile by 8) instead of all M tiles of 1-2 columns, so more of the activation stays in L2
  // (Qwen3-8B batch 16, 19-25 M tiles: 11.98 -> 11.60 ms per step; at 10 M tiles, 14B batch
  // 8, the grouping was 0.8% slower, so fewer stay in plain M-fastest order).
  constexpr int GM = 8;
  if (MT >= 2 * GM) {
    const int grp = L / (GM * NT), first = grp * GM;
    const int gm = min(MT - first, GM), r = L - grp * GM * NT;
    mt = first + r % gm;
    nt = r / gm;
    return;
  }
  mt = L % MT;
  nt = L / MT;
}

// Base pointer of tile-local B row `lr` of N tile `nt` (B rows may come from segments).
template <typename TB, int BN, int EPI>
__device__ __forceinline__ const TB* b_row(const GemmArgs& a, int nt, int lr, bool& ok) {
  if (EPI == EPI_SWIGLU) {
    constexpr int half = BN / 2;
    const int f = nt * half + (lr % half);
    ok = f < a.N;
    const TB* base = (const TB*)(lr < half ? a.B0 : a.B1);
    return base + (int64_t)(ok ? f : 0) * a.K;
  } else {
    int n = nt * BN + lr;
    ok = n < a.N;
    if (!ok) n = 0;
    if (a.seg_rows > 0) {
      const int si = n / a.seg_rows;
      return (const TB*)a.seg[si] + (int64_t)(n - si * a.seg_rows) * a.K;
    }
    if (n < a.n1) return (const TB*)a.B0 + (int64_t)n * a.K;
    if (n < a.n2) return (const TB*)a.B1 + (int64_t)(n - a.n1) * a.K;
    return (const TB*)a.B2 + (int64_t)(n - a.n2) * a.K;
  }
}

// LDS row of B fragment ni for wave column wn.  SwiGLU tiles hold BN/2 gate rows then
// BN/2 up rows; each wave takes the same FFN columns from both halves so that gate and
// up of one output land in the same thread.
template <int BN, int WN, int FN, int EPI>
__device__ __forceinline__ int b_frag_row(int wn, int ni) {
  if (EPI == EPI_SWIGLU) {
    return ni < FN / 2 ? wn * (WN / 2) + ni * 16 : BN / 2 + wn * (WN / 2) + (ni - FN / 2) * 16;
  }
  return wn * WN + ni * 16;
}

// SwiGLU outputs of a tile, staged in LDS (rows [0, BM) x OC columns, row stride LDO), leave
// as 16-byte row pieces instead of one 2-byte store per accumulator element.
template <int BM, int OC, int LDO>
__device__ __forceinline__ void swiglu_copy_out(const bf16_t* so, bf16_t* C, int64_t ldc, int m0, int f0, int M,
                                                int N) {
  static_assert(OC % 8 == 0 && LDO % 8 == 0, "16-byte pieces");
  constexpr int CPR = OC / 8;
  for (int e = threadIdx.x; e < BM * CPR; e += blockDim.x) {
    const int lrow = e / CPR, ch = e % CPR;
    const int row = m0 + lrow, f = f0 + ch * 8;
    if (row >= M || f >= N) continue;
    const bf16_t* src = so + lrow * LDO + ch * 8;
    bf16_t* dst = C + (int64_t)row * ldc + f;
    if (f + 8 <= N && (ldc & 7) == 0) {
      *(uint4*)dst = *(const uint4*)src;
    } else {
      for (int j = 0; j < 8 && f + j < N; ++j) dst[j] = src[j];
    }
  }
}

// ------------------------------------------------------------------ pipelined bf16 path
// Tiles stream through a ring of STAGES LDS buffers filled by direct global->LDS DMA
// (global_load_lds_dwordx4: lane i's 16 bytes land at M0 + 16*i, so one instruction moves
// 1 KB = 1024/BKB rows of a tile).  A row's 16-byte chunk c is stored in slot
// c ^ swizzle(row) so that the MFMA fragment reads (16 rows, same chunk) spread over the LDS
// banks.  Each wave waits only for its own DMA of the stage it is about to read (vmcnt
// counts outstanding DMA instructions), then one s_barrier makes every wave's part of that
// stage visible; the refill of the ring slot freed by the previous iteration is issued
// right after the barrier, so STAGES-1 stages are in flight while one is consumed.
// Cache policy of the weight DMA: when the grid has one M tile every weight element is read by
// exactly one workgroup, so the weights stream through L2 as non-temporal lines (nt) and leave
// the activation tile, which every workgroup re-reads, resident (M <= 320: 3-7% per GEMM); with
// several M tiles the weight tiles are shared and keep the default policy.
constexpr int kAuxStream = 2;
template <int AUX>
__device__ __forceinline__ void dma16(const void* g, void* l) {
  __builtin_amdgcn_global_load_lds(g, (lds_void_t*)l, 16, 0, AUX);
}

template <int CH>
__device__ __forceinline__ int swz(int r, int c) {
  if (CH == 16 || CH == 32) return c ^ (r & 15);  // 16 rows of a fragment read: 16 distinct slots
  if (CH == 8) return c ^ (r & 7);
  return c ^ ((r >> 1) & 3);
}

// DUAL: A is given as two bf16 planes (hi at A, lo at A + a.lo_off elements) whose sum is
// the float32 operand; every weight fragment is multiplied by both planes.
template <int BM, int BN, int WMW, int WNW, int STAGES, int BKB, int EPI, int DUAL>
__global__ __launch_bounds__(64 * WMW * WNW) void gemm_pipe_kernel(GemmArgs a, int MT, int NT) {
  constexpr int NW = WMW * WNW;
  constexpr int NPL = DUAL ? 2 : 1;  // A planes
  constexpr int CH = BKB / 16;      // 16-byte chunks per tile row per stage
  constexpr int RPI = 1024 / BKB;   // tile rows per DMA instruction
  constexpr int KB = BKB / 2;       // bf16 elements per tile row per stage
  constexpr int WM = BM / WMW, WN = BN / WNW;
  constexpr int FM = WM / 16, FN = WN / 16;
  constexpr int A_INS = NPL * BM / RPI / NW, B_INS = BN / RPI / NW;
  static_assert(A_INS * RPI * NW == NPL * BM && B_INS * RPI * NW == BN, "tile rows must split evenly over waves");
  static_assert(KB % 32 == 0, "stage depth must be a multiple of the MFMA k");
  constexpr int A_ROWS = NPL * BM;   // stage rows of A: [0, BM) hi (or the only plane), [BM, 2BM) lo
  constexpr int STAGE_BYTES = (A_ROWS + BN) * BKB;
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];

  if (a.only_if && *a.only_if == 0) return;
  // Split-K: the S splits of one output tile are consecutive logical workgroups; split s
  // covers K range [s*K/S, (s+1)*K/S) and stores into plane s of C.
  const int S = a.splits;
  int mt, nt;
  tile_of(blockIdx.x / S, MT, NT, mt, nt);
  const int split = blockIdx.x % S;
  const int Ks = a.K / S, kbeg = split * Ks;
  const int m0 = mt * BM;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WNW, wn = wave % WNW;

  // Per-lane DMA sources.  Rows past M or N are clamped to the last valid row: their
  // products land in accumulator rows/columns that the epilogue never stores.
  const bf16_t* asrc[A_INS];
  const bf16_t* bsrc[B_INS];
  const int lrow = lane / CH, lslot = lane % CH;
#pragma unroll
  for (int j = 0; j < A_INS; ++j) {
    const int r = (wave + NW * j) * RPI + lrow;   // stage row
    const int plane = r >= BM ? 1 : 0;
    const int gm = min(m0 + r - plane * BM, a.M - 1);
    asrc[j] = (const bf16_t*)a.A + (plane ? a.lo_off : 0) + (int64_t)gm * a.lda + kbeg + swz<CH>(r, lslot) * 8;
  }
#pragma unroll
  for (int j = 0; j < B_INS; ++j) {
    const int r = (wave + NW * j) * RPI + lrow;
    bool ok;
    bsrc[j] = b_row<bf16_t, BN, EPI>(a, nt, r, ok) + kbeg + swz<CH>(r, lslot) * 8;
  }
  auto issue = [&](int kt, int stage) {
    unsigned char* sb = smem + stage * STAGE_BYTES;
    const int k0 = kt * KB;
#pragma unroll
    for (int j = 0; j < A_INS; ++j)
      __builtin_amdgcn_global_load_lds((const void*)(asrc[j] + k0), (lds_void_t*)(sb + (wave + NW * j) * 1024), 16, 0, 0);
    if (MT == 1) {
#pragma unroll
      for (int j = 0; j < B_INS; ++j) dma16<kAuxStream>(bsrc[j] + k0, sb + A_ROWS * BKB + (wave + NW * j) * 1024);
    } else {
#pragma unroll
      for (int j = 0; j < B_INS; ++j) dma16<0>(bsrc[j] + k0, sb + A_ROWS * BKB + (wave + NW * j) * 1024);
    }
  };

  f32x4_t acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  const int KT = Ks / KB;
  const int lr = lane & 15, lc = lane >> 4;
  debug_poison_lds<STAGES * STAGE_BYTES>(smem);
  // Fragments of k-step ks (32 deep) of the stage in ring slot `slot`.
  auto load_frags = [&](int slot, int ks, bf16x8_t(&af)[NPL][FM], bf16x8_t(&bf)[FN]) {
    const unsigned char* sa = smem + slot * STAGE_BYTES;
    const unsigned char* sb = sa + A_ROWS * BKB;
    const int c = ks * 4 + lc;
#pragma unroll
    for (int ni = 0; ni < FN; ++ni) {
      const int r = b_frag_row<BN, WN, FN, EPI>(wn, ni) + lr;
      bf[ni] = *(const bf16x8_t*)(sb + r * BKB + swz<CH>(r, c) * 16);
    }
#pragma unroll
    for (int pl = 0; pl < NPL; ++pl)
#pragma unroll
      for (int mi = 0; mi < FM; ++mi) {
        const int r = pl * BM + wm * WM + mi * 16 + lr;
        af[pl][mi] = *(const bf16x8_t*)(sa + r * BKB + swz<CH>(r, c) * 16);
      }
  };
  // Row blocks wholly past M (wave-uniform) skip their products: a 17-row call on a 64-row
  // tile computes two blocks, not four.
  const int live_mi = min(FM, max(0, (a.M - m0 - wm * WM + 15) / 16));
  auto mfmas = [&](const bf16x8_t(&af)[NPL][FM], const bf16x8_t(&bf)[FN]) {
#pragma unroll
    for (int pl = 0; pl < NPL; ++pl)
#pragma unroll
      for (int mi = 0; mi < FM; ++mi) {
        if (mi >= live_mi) continue;
#pragma unroll
        for (int ni = 0; ni < FN; ++ni)
          acc[mi][ni] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[pl][mi], bf[ni], acc[mi][ni], 0, 0, 0);
      }
  };
  bf16x8_t af[2][NPL][FM], bfr[2][FN];  // two register sets, declared once for the whole loop
#pragma unroll
  for (int st = 0; st < STAGES - 1; ++st)
    if (st < KT) issue(st, st);
  for (int kt = 0; kt < KT; ++kt) {
    if (kt + STAGES - 2 < KT) wait_vmcnt<(STAGES - 2) * (A_INS + B_INS)>();
    else wait_vmcnt<0>();
    __builtin_amdgcn_s_barrier();
    if (kt + STAGES - 1 < KT) issue(kt + STAGES - 1, (kt + STAGES - 1) % STAGES);
    // Fragments of k-step ks+1 are read from LDS before k-step ks's MFMAs are issued (two
    // register sets), so the LDS latency hides behind the math.
    load_frags(kt % STAGES, 0, af[0], bfr[0]);
#pragma unroll
    for (int ks = 0; ks < KB / 32; ++ks) {
      const int cur = ks & 1;
      if (ks + 1 < KB / 32) load_frags(kt % STAGES, ks + 1, af[cur ^ 1], bfr[cur ^ 1]);
      __builtin_amdgcn_sched_barrier(0);  // keep the prefetch ahead of this step's MFMAs
      mfmas(af[cur], bfr[cur]);
    }
  }

  if constexpr (EPI == EPI_QKV) {
    // One 128-wide head per wave column: the row's sum of squares over the head is this
    // lane's eight columns plus the 16 lanes sharing the row (DPP), and RoPE's rotate-half
    // partner of column d (d +- 64) is fragment ni +- 4 of the same lane.  Same arithmetic as
    // the q/k-norm kernel: y = x * (1 / sqrt(ss / 128 + eps)) * g, then
    // y_d = y_d cos - y_{d+64} sin, y_{d+64} = y_{d+64} cos + y_d sin.  The bf16 results go
    // through this wave's part of the (now free) LDS ring, [WM rows][128 + 8 columns], so that
    // Q and K leave as 16-byte row pieces and V^T as 64 consecutive rows per store (the launch
    // sizes the dynamic LDS for this staging: up to 139 KB against the 128 KB ring).
    static_assert(WN == 128 && FN == 8 && WM <= 64 && DUAL == 0, "one 128-wide head per wave column");
    constexpr int LDT = 136;  // staging row stride in bf16 (272 bytes: rows fall on different banks)
    const QkvEpi& e = a.qkv;
    const int slot = nt * (BN / 128) + wn;
    const int grp = e.n_q / e.n_kv;
    const bool live = slot < e.n_q + 2 * e.n_kv;
    const bool isv = slot >= e.n_q + e.n_kv, isq = slot < e.n_q;
    bf16_t* stg = (bf16_t*)smem + wave * WM * LDT;
    __syncthreads();  // every wave is done with the ring
    if (!live) return;  // past the last head (no barrier follows)
    const float* gain = isq ? e.qn : e.kn;
    const int row0 = m0 + wm * WM;  // this wave's first row
#pragma unroll
    for (int mi = 0; mi < FM; ++mi) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int lrow = mi * 16 + lc * 4 + r, row = row0 + lrow;
        float v[FN];
#pragma unroll
        for (int ni = 0; ni < FN; ++ni) v[ni] = acc[mi][ni][r];
        if (!isv) {
          if (e.qk_norm) {
            float ss = 0.f;
#pragma unroll
            for (int ni = 0; ni < FN; ++ni) ss += v[ni] * v[ni];
            ss = row16_sum(ss);
            const float rn = 1.0f / sqrtf(ss / 128.0f + e.eps);
#pragma unroll
            for (int ni = 0; ni < FN; ++ni) v[ni] = v[ni] * rn * gain[ni * 16 + lr];
          }
          const int rc = min(row, a.M - 1), b = rc / e.R;
          const float2* cs = e.table + ((int64_t)b * (2 * e.gamma + 1) + row_pos_offset(rc - b * e.R, e.gamma)) * 64 + lr;
#pragma unroll
          for (int ni = 0; ni < FN / 2; ++ni) {
            const float2 c = cs[ni * 16];
            const float lo = v[ni], hi = v[ni + 4];
            v[ni] = lo * c.x + -1.f * hi * c.y;
            v[ni + 4] = hi * c.x + 1.f * lo * c.y;
          }
        }
#pragma unroll
        for (int ni = 0; ni < FN; ++ni) stg[lrow * LDT + ni * 16 + lr] = f2bf(v[ni]);
      }
    }
    if (!isv) {
      // row pieces: lane (rq, piece) stores 16 bytes = columns 8 piece .. +7 of rows rq, rq+4, ...
      const int piece = lane & 15;
#pragma unroll 4
      for (int lrow = lane >> 4; lrow < WM; lrow += 4) {
        const int row = row0 + lrow;
        if (row >= a.M) break;
        const int b = row / e.R, rr = row - b * e.R;
        bf16_t* dst = isq ? (bf16_t*)e.Q + (((int64_t)(b * e.n_kv + slot / grp) * grp + slot % grp) * e.R + rr) * 128
                          : (bf16_t*)e.Kb + ((int64_t)(b * e.n_kv + (slot - e.n_q)) * e.Rp + rr) * 128;
        *(uint4*)(dst + piece * 8) = *(const uint4*)(stg + lrow * LDT + piece * 8);
      }
    } else {
      // V^T [128][Rp]: lane = row, one store per head dimension (WM consecutive rows of a
      // request, split where a request ends)
      const int row = row0 + lane;
      if (lane < WM && row < a.M) {
        const int b = row / e.R, rr = row - b * e.R;
        bf16_t* dst = (bf16_t*)e.Vb + (int64_t)(b * e.n_kv + (slot - e.n_q - e.n_kv)) * 128 * e.Rp + rr;
        for (int d = 0; d < 128; ++d) dst[(int64_t)d * e.Rp] = stg[lane * LDT + d];
      }
    }
    return;
  }
  if constexpr (EPI == EPI_TOP2) {
    // One (key1, key2, third value) triple per row and 128-column tile (WPT wave columns each):
    // per lane over its columns of each row (FN of them); then the 16 lanes that share the
    // row (DPP); then the tile's wave columns through LDS, which the K loop no longer uses.
    static_assert(BN % 128 == 0 && 128 % WN == 0, "top-2 tiles are 128 columns of whole wave columns");
    constexpr int WPT = 128 / WN, QT = BN / 128;
    __syncthreads();
    Top3* xs = (Top3*)smem;  // [WNW][BM]
    // one 16-row block at a time (keeps few triples live beside the accumulators)
#pragma unroll
    for (int mi = 0; mi < FM; ++mi)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        Top3 t{};
#pragma unroll
        for (int ni = 0; ni < FN; ++ni) {
          const int col = nt * BN + wn * WN + ni * 16 + lr;
          if (col < a.N) t.add(argmax_key(acc[mi][ni][r], (uint32_t)col));
        }
        t = t.row16();
        if (lr == 0) xs[wn * BM + wm * WM + mi * 16 + (lane >> 4) * 4 + r] = t;
      }
    __syncthreads();
    const int n_tiles = (a.N + 127) / 128;
    for (int e = threadIdx.x; e < QT * BM; e += blockDim.x) {
      const int lrow = e % BM, q = e / BM;
      const int row = m0 + lrow, tile = nt * QT + q;
      if (row >= a.M || tile >= n_tiles) continue;
      Top3 m = xs[q * WPT * BM + lrow];
      for (int c = 1; c < WPT; ++c) m = Top3::merge(m, xs[(q * WPT + c) * BM + lrow]);
      uint64_t* o = (uint64_t*)a.C + ((int64_t)row * a.ldc + tile) * 3;
      o[0] = m.k1;
      o[1] = m.k2;
      o[2] = (uint64_t)__float_as_uint(m.v3);
    }
    return;
  }
  if constexpr (EPI == EPI_SWIGLU) {
    constexpr int OC = BN / 2, LDO = OC + 8;
    static_assert(BM * LDO * 2 <= STAGES * STAGE_BYTES, "the output tile fits the ring");
    bf16_t* so = (bf16_t*)smem;
    __syncthreads();  // every wave is done with the ring
#pragma unroll
    for (int mi = 0; mi < FM; ++mi)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int lrow = wm * WM + mi * 16 + (lane >> 4) * 4 + r;
#pragma unroll
        for (int ni = 0; ni < FN / 2; ++ni)
          so[lrow * LDO + wn * (WN / 2) + ni * 16 + lr] = f2bf(silu_f(acc[mi][ni][r]) * acc[mi][ni + FN / 2][r]);
      }
    __syncthreads();
    swiglu_copy_out<BM, OC, LDO>(so, (bf16_t*)a.C, a.ldc, m0, nt * OC, a.M, a.N);
    return;
  }
#pragma unroll
  for (int mi = 0; mi < FM; ++mi) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int row = m0 + wm * WM + mi * 16 + (lane >> 4) * 4 + r;
      if (row >= a.M) continue;
      if constexpr (EPI == EPI_STORE_BF16) {
        bf16_t* C = (bf16_t*)a.C + (int64_t)row * a.ldc;
#pragma unroll
        for (int ni = 0; ni < FN; ++ni) {
          const int col = nt * BN + wn * WN + ni * 16 + lr;
          if (col < a.N) C[col] = f2bf(acc[mi][ni][r]);
        }
      } else {
        float* C = (float*)a.C + ((int64_t)split * a.M + row) * a.ldc;
#pragma unroll
        for (int ni = 0; ni < FN; ++ni) {
          const int col = nt * BN + wn * WN + ni * 16 + lr;
          if (col < a.N) {
            if constexpr (EPI == EPI_ADD_F32) C[col] += acc[mi][ni][r];
            else C[col] = acc[mi][ni][r];
          }
        }
      }
    }
  }
}


// ------------------------------------------------------------------ float32 FMA path
// ------------------------------------------------------------ fragment-ordered A path
// For M <= 320 one 320-row tile covers every row, so each workgroup multiplies the whole
// activation operand with its own weight slice: A is re-read by every workgroup, the weights
// once.  A therefore bypasses LDS: it arrives in MFMA fragment order (frag_index), and each
// of the 4 waves (one per SIMD) loads the fragments of its own 80 rows straight into a
// register ring SB stages deep (one 16-byte load per lane per 1 KB block).  Only the weight
// tile (96 rows of B per 64-deep K step) goes through an LDS ring filled by direct DMA (as
// non-temporal lines: each is read once) and read by all four waves.  Row blocks past the last valid one are clamped to it (their
// accumulator rows are never stored).  SwiGLU tiles hold 48 gate + 48 up columns; the fp32
// store splits K over `splits` workgroups writing planes [S][M][ldc].
template <int EPI, int SB, int SKIP>
__global__ __launch_bounds__(256) void gemm_adir_kernel(GemmArgs a, int NT) {
  constexpr int BM = 320, BN = 96, BKB = 128, KB = 64, KS = KB / 32, CH = BKB / 16, RPI = 1024 / BKB;
  constexpr int NW = 4, WM = BM / NW, FM = WM / 16, FN = BN / 16;
  constexpr int B_INS = BN / RPI / NW;
  constexpr int STAGE_BYTES = BN * BKB;
  static_assert(B_INS * RPI * NW == BN, "weight rows must split evenly over waves");
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];

  const int S = a.splits;
  int mt, nt;
  tile_of(blockIdx.x / S, 1, NT, mt, nt);
  const int split = blockIdx.x % S;
  const int Ks = a.K / S, kbeg = split * Ks;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int lr = lane & 15, lc = lane >> 4;

  const int KC = a.K / 32, last_rb = (a.M - 1) >> 4;
  const bf16_t* ap[FM];
#pragma unroll
  for (int mi = 0; mi < FM; ++mi) {
    const int rb = min(wave * FM + mi, last_rb);
    ap[mi] = (const bf16_t*)a.A + ((int64_t)rb * KC + kbeg / 32) * 512 + (lane & 15) * 32 + (lane >> 4) * 8;
  }
  const bf16_t* bsrc[B_INS];
  const int lrow = lane / CH, lslot = lane % CH;
#pragma unroll
  for (int j = 0; j < B_INS; ++j) {
    const int r = (wave + NW * j) * RPI + lrow;
    bool ok;
    bsrc[j] = b_row<bf16_t, BN, EPI>(a, nt, r, ok) + kbeg + swz<CH>(r, lslot) * 8;
  }

  bf16x8_t abuf[SB][KS][FM];
  // K step k_ld's A fragments into register slot `buf`, its weight tile into LDS slot `slot`
  auto issue = [&](int k_ld, int slot, int buf) {
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
#pragma unroll
      for (int mi = 0; mi < FM; ++mi)
        abuf[buf][ks][mi] = *(const bf16x8_t*)(ap[mi] + (int64_t)(k_ld * KS + ks) * 512);
    __builtin_amdgcn_sched_barrier(0);
    unsigned char* sb = smem + slot * STAGE_BYTES;
#pragma unroll
    for (int j = 0; j < B_INS; ++j) dma16<kAuxStream>(bsrc[j] + k_ld * KB, sb + (wave + NW * j) * 1024);
    __builtin_amdgcn_sched_barrier(0);
  };

  f32x4_t acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  // KT is a multiple of SB (host check).  Step kt's loads were issued SB-1 steps earlier;
  // past the end the refill repeats the last step into a slot nobody reads again.
  constexpr int PER = KS * FM + B_INS;  // vector memory instructions per issue
  const int KT = Ks / KB;
  debug_poison_lds<SB * STAGE_BYTES>(smem);
#pragma unroll
  for (int s = 0; s < SB - 1; ++s) issue(s, s, s);
  for (int kt0 = 0; kt0 < KT; kt0 += SB) {
#pragma unroll
    for (int u = 0; u < SB; ++u) {
      const int kt = kt0 + u;
      wait_vmcnt<(SB - 2) * PER>();
      __builtin_amdgcn_s_barrier();
      const int nx = kt + SB - 1;
      issue(min(nx, KT - 1), nx % SB, (u + SB - 1) % SB);
      const unsigned char* sb = smem + (kt % SB) * STAGE_BYTES;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const int c = ks * 4 + lc;
        bf16x8_t bfr[FN];
#pragma unroll
        for (int ni = 0; ni < FN; ++ni) {
          const int r = b_frag_row<BN, BN, FN, EPI>(0, ni) + lr;
          bfr[ni] = *(const bf16x8_t*)(sb + r * BKB + swz<CH>(r, c) * 16);
        }
#pragma unroll
        for (int mi = 0; mi < FM; ++mi) {
          // SKIP: a row block past M (wave-uniform) has no products.  Only instantiated for short
          // calls: at 289 rows the branch between MFMA groups cost 9% (72 -> 78.5 us gate|up).
          if (SKIP && wave * FM + mi > last_rb) continue;
#pragma unroll
          for (int ni = 0; ni < FN; ++ni)
            acc[mi][ni] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(abuf[u][ks][mi], bfr[ni], acc[mi][ni], 0, 0, 0);
        }
      }
    }
  }
  wait_vmcnt<0>();

  if constexpr (EPI == EPI_SWIGLU) {
    constexpr int OC = BN / 2, LDO = OC + 8;
    static_assert(BM * LDO * 2 <= SB * STAGE_BYTES, "the output tile fits the ring");
    bf16_t* so = (bf16_t*)smem;
    __syncthreads();  // every wave is done with the ring
#pragma unroll
    for (int mi = 0; mi < FM; ++mi)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int lrow = wave * WM + mi * 16 + lc * 4 + r;
#pragma unroll
        for (int ni = 0; ni < FN / 2; ++ni)
          so[lrow * LDO + ni * 16 + lr] = f2bf(silu_f(acc[mi][ni][r]) * acc[mi][ni + FN / 2][r]);
      }
    __syncthreads();
    swiglu_copy_out<BM, OC, LDO>(so, (bf16_t*)a.C, a.ldc, 0, nt * OC, a.M, a.N);
    return;
  }
#pragma unroll
  for (int mi = 0; mi < FM; ++mi) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int row = wave * WM + mi * 16 + lc * 4 + r;
      if (row >= a.M) continue;
      {
        float* C = (float*)a.C + ((int64_t)split * a.M + row) * a.ldc;
#pragma unroll
        for (int ni = 0; ni < FN; ++ni) {
          const int col = nt * BN + ni * 16 + lr;
          if (col < a.N) C[col] = acc[mi][ni][r];
        }
      }
    }
  }
}

template <int EPI>
__global__ __launch_bounds__(256) void gemm_f32_kernel(GemmArgs a, int MT, int NT) {
  constexpr int BM = 64, BN = 64, BKF = 16;
  __shared__ float As[BKF][BM + 4];
  __shared__ float Bs[BKF][BN + 4];
  const int mt = blockIdx.x % MT, nt = blockIdx.x / MT;
  const int m0 = mt * BM;
  const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
  const int lrow = tid >> 2, lk = (tid & 3) * 4;
  bool bok;
  const float* bsrc = b_row<float, BN, EPI>(a, nt, lrow, bok);
  const float* A = (const float*)a.A;
  const int gm = m0 + lrow;
  float acc[4][4] = {};
  int cols[4];
#pragma unroll
  for (int j = 0; j < 4; ++j)
    cols[j] = (EPI == EPI_SWIGLU) ? (j < 2 ? tx * 2 + j : BN / 2 + tx * 2 + (j - 2)) : tx * 4 + j;
  for (int k0 = 0; k0 < a.K; k0 += BKF) {
    float4 va = gm < a.M ? *(const float4*)(A + (int64_t)gm * a.lda + k0 + lk) : make_float4(0, 0, 0, 0);
    float4 vb = bok ? *(const float4*)(bsrc + k0 + lk) : make_float4(0, 0, 0, 0);
    As[lk + 0][lrow] = va.x; As[lk + 1][lrow] = va.y; As[lk + 2][lrow] = va.z; As[lk + 3][lrow] = va.w;
    Bs[lk + 0][lrow] = vb.x; Bs[lk + 1][lrow] = vb.y; Bs[lk + 2][lrow] = vb.z; Bs[lk + 3][lrow] = vb.w;
    __syncthreads();
#pragma unroll
    for (int k = 0; k < BKF; ++k) {
      float av[4], bv[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) av[i] = As[k][ty * 4 + i];
#pragma unroll
      for (int j = 0; j < 4; ++j) bv[j] = Bs[k][cols[j]];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(av[i], bv[j], acc[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = m0 + ty * 4 + i;
    if (row >= a.M) continue;
    float* C = (float*)a.C + (int64_t)row * a.ldc;
    if constexpr (EPI == EPI_SWIGLU) {
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int f = nt * (BN / 2) + tx * 2 + j;
        if (f < a.N) C[f] = silu_f(acc[i][j]) * acc[i][j + 2];
      }
    } else {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int col = nt * BN + tx * 4 + j;
        if (col < a.N) {
          if constexpr (EPI == EPI_ADD_F32) C[col] += acc[i][j];
          else C[col] = acc[i][j];
        }
      }
    }
  }
}


template <int EPI>
hipError_t run_f32(const GemmArgs& a, hipStream_t st) {
  const int MT = (a.M + 63) / 64;
  const int NT = EPI == EPI_SWIGLU ? (a.N + 31) / 32 : (a.N + 63) / 64;
  hipLaunchKernelGGL((gemm_f32_kernel<EPI>), dim3(MT * NT), dim3(256), 0, st, a, MT, NT);
  return hipGetLastError();
}

template <int EPI>
hipError_t run_adir(const GemmArgs& a, hipStream_t st) {
  constexpr int SB = 4, BN = 96, lds = SB * BN * 128;
  static_assert(EPI == EPI_SWIGLU || EPI == EPI_STORE_F32, "fragment-ordered A: SwiGLU or fp32 store");
  if (a.M > 320 || a.K % 32) return hipErrorInvalidValue;
  if (a.splits < 1 || (a.splits > 1 && EPI != EPI_STORE_F32) || a.K % (a.splits * 64 * SB) != 0)
    return hipErrorInvalidValue;
  const int NT = EPI == EPI_SWIGLU ? (a.N + BN / 2 - 1) / (BN / 2) : (a.N + BN - 1) / BN;
  // Up to 240 rows at least the last wave's 80 rows are empty: skip the products of row blocks
  // past M (the 36-layer target verifying 17 rows a request: 5.75 -> 5.40 ms at batch 1).
  auto kern = a.M <= 240 ? gemm_adir_kernel<EPI, SB, 1> : gemm_adir_kernel<EPI, SB, 0>;
  static const hipError_t attr0 =
      hipFuncSetAttribute((const void*)gemm_adir_kernel<EPI, SB, 0>, hipFuncAttributeMaxDynamicSharedMemorySize, lds);
  static const hipError_t attr1 =
      hipFuncSetAttribute((const void*)gemm_adir_kernel<EPI, SB, 1>, hipFuncAttributeMaxDynamicSharedMemorySize, lds);
  if (attr0 != hipSuccess) return attr0;
  if (attr1 != hipSuccess) return attr1;
  hipLaunchKernelGGL(kern, dim3(NT * a.splits), dim3(256), lds, st, a, NT);
  return hipGetLastError();
}

template <int BM, int BN, int WMW, int WNW, int STAGES, int BKB, int EPI, int DUAL = 0>
hipError_t run_pipe(const GemmArgs& a, hipStream_t st) {
  const int MT = (a.M + BM - 1) / BM;
  const int NT = EPI == EPI_SWIGLU ? (a.N + BN / 2 - 1) / (BN / 2) : (a.N + BN - 1) / BN;
  constexpr int ring = STAGES * ((DUAL ? 2 : 1) * BM + BN) * BKB;
  constexpr int stage_out = EPI == EPI_QKV ? (BM / WMW) * WMW * WNW * 136 * 2 : 0;  // the QKV epilogue's staging
  constexpr int lds = ring > stage_out ? ring : stage_out;
  static_assert(lds <= 163840, "LDS ring exceeds 160 KB");
  auto kern = gemm_pipe_kernel<BM, BN, WMW, WNW, STAGES, BKB, EPI, DUAL>;
  static const hipError_t attr =
      hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, lds);
  if (attr != hipSuccess) return attr;
  // planes are float32 [S][M][ldc]: only the float32 store epilogue may split K
  if (a.splits < 1 || (a.splits > 1 && EPI != EPI_STORE_F32) || a.K % (a.splits * (BKB / 2)) != 0)
    return hipErrorInvalidValue;
  hipLaunchKernelGGL(kern, dim3(MT * NT * a.splits), dim3(64 * WMW * WNW), lds, st, a, MT, NT);
  return hipGetLastError();
}

// Tile choice for the bf16 projections (measured on MI355X at Qwen3-8B N/K):
//  M <= 320 : weight streaming.  One 320-row tile covers every row, so each weight tile is
//             read once; 8 waves (80x64 each), a 2-deep ring of 64-wide K steps (SwiGLU:
//             320x96 tiles of 4 waves, 80 x (48 gate + 48 up) each).  The
//             fp32-store GEMMs (QKV, O, down, append) split K so that about 256 workgroups
//             run; their consumers add the S partial planes (gemm_splits).
//  M <= 64 (the context append, up to gamma+1 rows per request) and 320 < M <= 1024:
//             64x128 tiles, 3-deep ring;
//  larger   : 256x256 tiles, 8 waves (128x64 per wave), 2-deep ring.
// Fraction of the last round of workgroups that has work (one workgroup per CU) for
// BM x 256 tiles: 192-row tiles are taken when they fill the rounds clearly better (the
// Qwen3-8B O / down projections at 4624 rows: 304 tiles = 1.19 rounds with 256 rows, 400 =
// 1.56 with 192, measured 11% faster on MI355X).
double round_fill(int M, int N, int BM) {
  const double w = (double)((M + BM - 1) / BM) * ((N + 255) / 256) / 256.0;
  return w / ceil(w);
}

template <int EPI>
hipError_t run_bf16(const GemmArgs& a, hipStream_t st) {
  if (a.M > 1024) {
    if constexpr (EPI == EPI_STORE_F32) {
      // Fewer than 192 tiles of 256 x 256 (under three quarters of one round, e.g. the
      // 2048-row feature fusion, 4096 columns: 128 tiles): 128 x 128 tiles at two workgroups
      // per CU fill the chip instead.
      if (a.splits == 1 && (int64_t)((a.M + 255) / 256) * ((a.N + 255) / 256) < 192)
        return run_pipe<128, 128, 2, 2, 2, 128, EPI>(a, st);
      // One weight matrix, no split-K: when the last round of BM x 256 tiles is at most 60%
      // full, the columns of that round go to a second launch of 128 x 128 tiles (two
      // workgroups per CU) and the first runs whole rounds only.  Measured on MI355X at
      // Qwen3-8B batch 16 (4624 rows, 400 tiles of 192 x 256 = 1.56 rounds): O 876 -> 858,
      // down 2404 -> 2342 us per step.
      const bool bm192 = round_fill(a.M, a.N, 192) > round_fill(a.M, a.N, 256) + 0.1;
      const int BMc = bm192 ? 192 : 256;
      const int MT = (a.M + BMc - 1) / BMc, NT = (a.N + 255) / 256, T = MT * NT;
      const int NT1 = (T / 256) * 256 / MT;  // 256-column tiles of the whole rounds
      if (a.splits == 1 && a.seg_rows == 0 && a.n1 >= a.N && T % 256 != 0 && T % 256 <= 256 * 6 / 10 && NT1 > 0 &&
          NT1 < NT) {
        GemmArgs head = a, tail = a;
        const int n0 = NT1 * 256;
        head.N = n0;
        tail.B0 = tail.B1 = tail.B2 = (const bf16_t*)a.B0 + (int64_t)n0 * a.K;
        tail.n1 = tail.n2 = a.N - n0;
        tail.C = (float*)a.C + n0;
        tail.N = a.N - n0;
        const hipError_t e = bm192 ? run_pipe<192, 256, 2, 4, 2, 128, EPI>(head, st)
                                   : run_pipe<256, 256, 2, 4, 2, 128, EPI>(head, st);
        if (e != hipSuccess) return e;
        return run_pipe<128, 128, 2, 2, 2, 128, EPI>(tail, st);
      }
    }
    if (EPI != EPI_SWIGLU && round_fill(a.M, a.N, 192) > round_fill(a.M, a.N, 256) + 0.1)
      return run_pipe<192, 256, 2, 4, 2, 128, EPI>(a, st);
    if constexpr (EPI == EPI_SWIGLU) {
      // When the 256 x 256 tiles leave a last round of workgroups at most half full, the FFN
      // columns of that round go to a second launch of 128 x 128 tiles (64 gate + 64 up
      // columns, two workgroups per CU), four times as many workgroups each a quarter of the
      // work: the first launch runs whole rounds only.  Measured on MI355X: 4.3% off the
      // Qwen3-14B batch-8 gate/up (5.3 rounds), 2.6% off Qwen3-8B batch 16 (7.1 rounds).
      const int MT = (a.M + 255) / 256, NT = (a.N + 127) / 128, T = MT * NT;
      const int NT1 = (T / 256) * 256 / MT;  // FFN column tiles of the whole rounds
      if (T % 256 != 0 && T % 256 <= 128 && NT1 > 0 && NT1 < NT) {
        GemmArgs head = a, tail = a;
        head.N = NT1 * 128;
        const int f0 = NT1 * 128;
        tail.B0 = (const bf16_t*)a.B0 + (int64_t)f0 * a.K;
        tail.B1 = (const bf16_t*)a.B1 + (int64_t)f0 * a.K;
        tail.C = (bf16_t*)a.C + f0;
        tail.N = a.N - f0;
        const hipError_t e = run_pipe<256, 256, 2, 4, 2, 128, EPI>(head, st);
        if (e != hipSuccess) return e;
        return run_pipe<128, 128, 2, 2, 2, 128, EPI>(tail, st);
      }
    }
    return run_pipe<256, 256, 2, 4, 2, 128, EPI>(a, st);
  }
  // up to 32 rows (a 17-row verification, the context append, the sampled head's scores): a
  // 32-row tile halves the activation rows each stage loads (target at batch 1: -1.2%)
  if (a.M <= 32 && EPI != EPI_SWIGLU) return run_pipe<32, 128, 2, 2, 3, 128, EPI>(a, st);
  if (a.M > 320 || (a.M <= 64 && EPI != EPI_SWIGLU)) return run_pipe<64, 128, 2, 2, 3, 128, EPI>(a, st);
  // SwiGLU up to 64 rows (a target verifying 17 rows a request): weight streaming with a
  // 3-deep ring of 96-row weight tiles 128 deep in K (256-byte runs of each weight row) and 64
  // activation rows, four waves of 16 rows, the empty row blocks skipped.  36-layer target at
  // batch 1: gate|up 54 -> 46 us per layer with 64-deep stages in a 6-deep ring, then 1.2% off
  // the whole target with the 128-deep stages.
  if constexpr (EPI == EPI_SWIGLU)
    if (a.M <= 64) return run_pipe<64, 96, 4, 1, 3, 256, EPI>(a, st);
  // SwiGLU: 48 gate + 48 up rows per tile, so that the Qwen3-8B FFN (12288) gives 256 tiles
  if constexpr (EPI == EPI_SWIGLU) return run_pipe<320, 96, 4, 1, 2, 128, EPI>(a, st);
  return run_pipe<320, 128, 4, 2, 2, 128, EPI>(a, st);
}

}  // namespace

int gemm_splits(int amode, int epi, int M, int N, int K) {
  if (amode == A_BF16_FRAG) {
    // 96-column tiles; K steps of each split a multiple of the 4-deep ring
    if (epi != EPI_STORE_F32) return 1;
    const int NT = (N + 95) / 96;
    int S = 1;
    while (S < 16 && NT * S * 2 <= 256 && K % (256 * S * 2) == 0) S *= 2;
    return S;
  }
  if (amode != A_BF16 || epi != EPI_STORE_F32 || M > 320) return 1;
  const int NT = (N + 127) / 128;
  const int max_wg = M <= 64 ? 512 : 256;  // the M <= 64 tile fits two workgroups per CU
  int S = 1;
  while (S < 16 && NT * S * 2 <= max_wg && K % (64 * S * 2) == 0 && K / (S * 2) >= 256) S *= 2;
  return S;
}

hipError_t launch_gemm(int amode, int epi, const GemmArgs& a, hipStream_t st) {
  if (a.M <= 0 || a.N <= 0) return hipSuccess;
  if (a.seg_rows < 0 || (a.seg_rows > 0 && (epi == EPI_SWIGLU || a.N > kMaxGemmSegs * a.seg_rows)))
    return hipErrorInvalidValue;
  if (a.splits < 1) return hipErrorInvalidValue;
  if (a.splits > 1 && amode != A_BF16 && amode != A_BF16_FRAG) return hipErrorInvalidValue;
  if (amode == A_F32) {
    switch (epi) {
      case EPI_STORE_F32: return run_f32<EPI_STORE_F32>(a, st);
      case EPI_ADD_F32: return run_f32<EPI_ADD_F32>(a, st);
      case EPI_SWIGLU: return run_f32<EPI_SWIGLU>(a, st);
      default: return hipErrorInvalidValue;
    }
  }
  if (amode == A_BF16_DUAL) {
    if (epi == EPI_TOP2) return hipErrorInvalidValue;
    // 16 rows (the LM head over one request's gamma rows): 256-deep K stages (512-byte runs of
    // each embedding row) in a 2-deep ring of 160 KB, one workgroup per CU.  Measured on MI355X
    // for the whole batch-1 head: 64-deep stages at two workgroups per CU 280 us, 128-deep in a
    // 4-deep ring 266-270, 256-deep 256-258.  The per-32-deep-chunk order of the MFMAs (hi,
    // then lo) is unchanged.
    if (a.M <= 16) return run_pipe<16, 128, 1, 4, 2, 512, EPI_STORE_F32, 1>(a, st);
    // 32 rows (two requests): the same 128-deep stages in a 3-deep ring, 15% faster than the
    // 64-row tile with half its rows idle (batch-2 head 325-345 -> 282 us on MI355X).
    if (a.M <= 32) return run_pipe<32, 128, 1, 4, 3, 256, EPI_STORE_F32, 1>(a, st);
    if (a.M <= 64) return run_pipe<64, 128, 2, 2, 3, 128, EPI_STORE_F32, 1>(a, st);
    // 129-256 rows (batch 9-16): one 256-row tile (both planes, 2-deep ring of 160 KB), so each
    // weight tile is read once: the batch-16 head 860 -> 797 us.
    if (a.M > 128 && a.M <= 256) return run_pipe<256, 128, 4, 2, 2, 128, EPI_STORE_F32, 1>(a, st);
    return run_pipe<128, 128, 4, 2, 3, 128, EPI_STORE_F32, 1>(a, st);
  }
  if (epi == EPI_QKV) {
    if (amode != A_BF16 || a.M <= 1024 || a.splits != 1 || a.N != (a.qkv.n_q + 2 * a.qkv.n_kv) * 128 ||
        a.qkv.n_kv < 1 || a.qkv.n_q % a.qkv.n_kv || a.qkv.R < 1 || a.qkv.Rp < a.qkv.R)
      return hipErrorInvalidValue;
    // the same tile choice as the plain projection (192 rows when they fill the rounds better)
    if (round_fill(a.M, a.N, 192) > round_fill(a.M, a.N, 256) + 0.1)
      return run_pipe<192, 256, 4, 2, 2, 128, EPI_QKV, 0>(a, st);
    return run_pipe<256, 256, 4, 2, 2, 128, EPI_QKV, 0>(a, st);
  }
  if (epi == EPI_TOP2) {
    // Top-2 over every branch row from one bf16 plane.  Measured on MI355X at the Qwen3
    // vocabulary (272 rows a request): up to 1536 rows 192 x 128 tiles (4 waves of 96 x 64, a
    // 2-deep ring of 80 KB), 22% faster than the large-M tile at 272 rows and 10% at 1088;
    // beyond, the large-M tile (256 x 256, 8 waves of 128 x 64, two top-2 tiles per
    // workgroup), 12% faster at 4352 rows.
    if (amode != A_BF16 || a.ldc < (a.N + 127) / 128) return hipErrorInvalidValue;
    // exactly 193-256 rows (the greedy head's ranking at batch 13-16): one 256 x 256 tile row
    // (the batch-16 head 587 -> 526 us against two 192-row tiles)
    if (a.M > 192 && a.M <= 256) return run_pipe<256, 256, 2, 4, 2, 128, EPI_TOP2, 0>(a, st);
    if (a.M <= 1536) return run_pipe<192, 128, 2, 2, 2, 128, EPI_TOP2, 0>(a, st);
    return run_pipe<256, 256, 2, 4, 2, 128, EPI_TOP2, 0>(a, st);
  }
  if (amode == A_BF16_FRAG) {
    if (epi == EPI_SWIGLU) return run_adir<EPI_SWIGLU>(a, st);
    if (epi == EPI_STORE_F32) return run_adir<EPI_STORE_F32>(a, st);
    return hipErrorInvalidValue;
  }
  if (amode != A_BF16) return hipErrorInvalidValue;
  switch (epi) {
    case EPI_STORE_BF16: return run_bf16<EPI_STORE_BF16>(a, st);
    case EPI_STORE_F32: return run_bf16<EPI_STORE_F32>(a, st);
    case EPI_ADD_F32: return run_bf16<EPI_ADD_F32>(a, st);
    default: return run_bf16<EPI_SWIGLU>(a, st);
  }
}

}  // namespace dpara
