// Host-side launchers shared between the DPara translation units.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "common.h"

namespace dpara {

// Per-phase tracing: when enabled (dpara_profile_enable), records a HIP event pair on `st`
// around the scope.  A no-op otherwise.
struct Phase {
  Phase(const char* name, hipStream_t st);
  ~Phase();
  Phase(const Phase&) = delete;
  Phase& operator=(const Phase&) = delete;
  int slot;
  hipStream_t st;
};

// ---------------------------------------------------------------- GEMM
// C[M, N] (op)= A[M, K] . B[N, K]^T with B given in up to three row segments
// (rows [0, n1) from B0, [n1, n2) from B1, [n2, N) from B2), or, with seg_rows > 0 (not for
// EPI_SWIGLU), in equal segments: row n from seg[n / seg_rows], row n % seg_rows.
enum GemmEpi { EPI_STORE_F32 = 0, EPI_ADD_F32 = 1, EPI_SWIGLU = 2, EPI_STORE_BF16 = 3, EPI_TOP2 = 4, EPI_QKV = 5 };

// Parameters of the EPI_QKV epilogue: the Q|K|V projection of R rows per request written as
// the attention kernel's bf16 operands (Q [B, n_kv, grp * R, 128], in-block K [B, n_kv, Rp, 128],
// V^T [B, n_kv, 128, Rp]) after the per-head q/k RMSNorm (qk_norm != 0, gains qn / kn) and RoPE
// (table: (cos, sin) per request, position offset and frequency, as the q/k-norm kernel reads it).
struct QkvEpi {
  int R = 0, Rp = 0, gamma = 0, n_q = 0, n_kv = 0, qk_norm = 0;
  float eps = 0.f;
  const float* qn = nullptr;
  const float* kn = nullptr;
  const float2* table = nullptr;
  void* Q = nullptr;
  void* Kb = nullptr;
  void* Vb = nullptr;
};
// A_BF16: A is bf16, row-major with leading dimension lda.  A_F32: float32 FMA kernel
// (the float32 model path; B is then float32 too).
// A_BF16_DUAL: A given as two bf16 planes hi (at A) and lo (at A + lo_off elements) with
// hi + lo = the float32 operand to ~16 significant bits; both planes meet every weight tile.
// A_BF16_FRAG: A is bf16 in MFMA fragment order (frag_index; lda unused), M <= 320,
// K a multiple of 256 * splits; EPI_SWIGLU or EPI_STORE_F32 only.
enum GemmAMode { A_BF16 = 0, A_BF16_FRAG = 1, A_F32 = 2, A_BF16_DUAL = 3 };

// Element (row, k) of a bf16 operand stored in MFMA fragment blocks: blocks of 16 rows x 32 k
// (ceil(rows/16) x K/32 of them, row blocks outermost), row-major inside a block (64 bytes a
// row).  One wave loads one block (1 KB) with one 16-byte load per lane, lane l taking row
// l%16, k 8*(l/16) .. +7: the operand layout of v_mfma_f32_16x16x32_bf16.  A row's 32 values
// of a block are contiguous, so the writer (one row per workgroup) stores whole 64-byte pieces.
__host__ __device__ inline int64_t frag_index(int row, int k, int K) {
  return ((int64_t)(row >> 4) * (K >> 5) + (k >> 5)) * 512 + (row & 15) * 32 + (k & 31);
}

struct GemmArgs {
  const void* A;
  int64_t lda;
  const void* B0;
  const void* B1;
  const void* B2;
  int n1, n2;
  int M, N, K;
  void* C;
  int64_t ldc;
  int64_t lo_off;  // A_BF16_DUAL only
  int splits = 1;  // split-K: S >= 1 fp32 planes of C (plane stride M*ldc); EPI_STORE_F32 only
  // EPI_SWIGLU: B0 = gate [N, K], B1 = up [N, K], C = bf16/f32 [M, N] of silu(g) * u,
  // where N is the FFN width.
  // EPI_TOP2 (A_BF16 only): instead of C, per row and 128-column tile t the two largest
  // (value, column) argmax keys of the row's tile and the third largest value, as three
  // uint64 words at C + (row * ldc + t) * 3 (the value's float bits in the low word);
  // columns past N do not count.  ldc >= ceil(N / 128).
  const int* only_if = nullptr;  // non-NULL: every workgroup returns at once unless *only_if != 0
  int seg_rows = 0;               // > 0: B rows from seg[] (N <= kMaxGemmSegs * seg_rows)
  const void* seg[16] = {};
  QkvEpi qkv{};  // EPI_QKV only (bf16, head_dim 128, more than 1024 rows, no split-K)
};

constexpr int kMaxGemmSegs = 16;
hipError_t launch_gemm(int amode, int epi, const GemmArgs& a, hipStream_t st);
// Split-K factor launch_gemm uses for a bf16 fp32-store GEMM of this shape (1 = no split).
// The consumer of C sums the S planes in order 0..S-1.
int gemm_splits(int amode, int epi, int M, int N, int K);

// ---------------------------------------------------------------- attention
struct AttnArgs {
  int B, R, gamma, n_q, n_kv, hd;
  const void* Q;    // [B, n_kv, grp*R, hd] (row index g*R + row for query head kvh*grp + g)
  const void* Kb;   // [B, n_kv, Rp, hd]    in-block keys (rows R..Rp-1 unused)
  const void* Vb;   // [B, n_kv, hd, Rp]    in-block values, transposed (row stride Rp)
  int Rp;           // R rounded up to a multiple of 64
  const void* Kc;   // context K cache of this layer  [batch_cap, n_kv, cap, hd]
  const void* Vc;   // context V cache of this layer  [batch_cap, n_kv, hd, cap]
  int cap;
  const int* ctx_len;  // [B] device
  int S, chunk;        // bf16: keys split over S workgroups; float32: S == 1, chunk == cap
  float* Opart;        // [B, n_q, R, S, hd]
  float* MLpart;       // [B, n_q, R, S, 2]  (running max in log2 units, running sum)
  void* O;             // [B*R, n_q*hd]
  int spine_only;      // 1: rows are only the causal spine (no branches)
};
hipError_t launch_attention(int dtype, const AttnArgs& a, hipStream_t st);
// Largest key split S of the bf16 path (the fold kernel holds every partial of a row in
// registers).
constexpr int kMaxAttnSplits = 16;
int attn_rows_per_workgroup();  // query rows (over the heads of a KV group) per bf16 workgroup

// ---------------------------------------------------------------- elementwise
// Y[m] = rmsnorm(x) * g with x = X[in_row(m)] + sum_{s<S} P[s][in_row(m)] (P planes share
// X's layout, plane stride pstride floats), in_row(m) = (m / grp) * in_stride + in_off + m % grp.
// write_back: also store x into X (folds the pending partial sums into the residual stream).
hipError_t launch_rmsnorm(int out_dtype, int rows, int H, float* X, int grp, int64_t in_stride,
                          int in_off, const float* P, int S, int64_t pstride, int write_back,
                          const float* g, float eps, void* Y, hipStream_t st);
// The same with Y written as bf16 in MFMA fragment order (frag_index, K = H; rows past
// `rows` in the last 16-row block are left untouched).  H a multiple of 32.
hipError_t launch_rmsnorm_frag(int rows, int H, float* X, const float* P, int S, int64_t pstride,
                               const float* g, float eps, void* Y, hipStream_t st);
// The backbone input rows (spine rows: their tokens' embeddings; mask rows: the mask embedding)
// and the RoPE table of positions ctx_len .. ctx_len + n_pos - 1, in one launch
hipError_t launch_assemble_rows_rope(int dtype, int B, int R, int gamma, int H, int V, const int* spine,
                                     const void* embed, const void* mask_emb, float* X, int* status, int n_pos,
                                     int hd, float base, const int* ctx_len, float2* table, hipStream_t st);
hipError_t launch_rope_table(int B, int n_pos, int hd, float base, const int* ctx_len,
                             int pos_off, float2* table, hipStream_t st);
// QKV: S fp32 planes [S][B*R][(n_q+2n_kv)*hd], summed in order.
hipError_t launch_qk_norm_rope(int dtype, int B, int R, int Rp, int gamma, int n_q, int n_kv, int hd,
                               int qk_norm, float eps, const float* QKV, int S, const float* qn,
                               const float* kn, const float2* table, void* Q, void* Kb,
                               void* Vb, hipStream_t st);
hipError_t launch_gather_feats(int dtype, int B, int CH, int c0, int n_max, int H,
                               const void* feats, void* F, hipStream_t st);
// K/V of the appended rows for nl consecutive layers: KV holds S fp32 planes
// [S][B*CH][nl][2*n_kv*hd] (layer j's K then V entries), summed in order; layer j uses
// kn[j] and writes the caches at Kc/Vc + j * layer_elems.
// rope: [B*CH][hd/2] (cos, sin) of row m's position max(ctx_len[b], 0) + c0 + (m % CH).
constexpr int kMaxAppendLayers = 8;
struct KvLayers {
  const float* kn[kMaxAppendLayers];
};
hipError_t launch_kv_store(int dtype, int B, int CH, int c0, int n_max, int n_kv, int hd,
                           int qk_norm, float eps, const float2* rope, const float* KV, int S,
                           int nl, const KvLayers& kn, const int* n_new, const int* ctx_len, int cap,
                           void* Kc, void* Vc, size_t layer_elems, int* status, hipStream_t st);
// out[m * n_out + j][0..H) = X[m] + sum_{s<S} P[s][m] for rows m < rows, rounded to bf16
// (out_f32 == 0) or kept float32.
hipError_t launch_emit_hidden(int rows, int H, const float* X, const float* P, int S, int64_t pstride, void* out,
                              int n_out, int j, hipStream_t st, int out_f32 = 0);
hipError_t launch_ctx_len_update(int B, int n_max, int cap, const int* n_new, int* ctx_len,
                                 int* status, hipStream_t st);
hipError_t launch_clear_status(int* status, hipStream_t st);

// ---------------------------------------------------------------- verify / head
// Sampled head (sampling variant): with on != 0 every head step scores s = z * inv_t, writes
// s to scores[b][step-1][v] when scores is non-NULL, and ranks s + Gumbel(key; head tag, b,
// step, v) instead of z; margins are then those of the perturbed scores.
// The generator's key is (k0, k1), or the 64-bit seed at seed_dev read when the kernel runs
// (so a captured graph can draw a fresh seed per replay).
struct Sampling {
  int on;
  float inv_t;
  uint32_t k0, k1;
  const uint64_t* seed_dev;
  float* scores;
};
__device__ __forceinline__ void sampling_key(const Sampling& s, uint32_t& k0, uint32_t& k1) {
  if (s.seed_dev) {
    const uint64_t v = *s.seed_dev;
    k0 = (uint32_t)v;
    k1 = (uint32_t)(v >> 32);
  } else {
    k0 = s.k0;
    k1 = s.k1;
  }
}
hipError_t launch_verify(int logits_dtype, int B, int gamma, int V, const void* logits,
                         const int* spine, int* accept_len, int* bonus, int* target_argmax,
                         uint64_t* part, int n_chunks, int chunk, int* status, hipStream_t st);
// Speculative-sampling verification (sampling variant): per request, the logsumexp of every
// target row (scaled by inv_t) and draft-score row in vocabulary chunks, one wave for the
// acceptance test of each draft, then the bonus drawn by Gumbel-max from the residual
// max(0, p_r - q_{r+1}) (from p_r if rounding leaves it empty) or, after full acceptance,
// from p_gamma.  verify_sampled_bytes gives the scratch bytes it needs.
size_t verify_sampled_bytes(int B, int gamma, int n_chunks);
hipError_t launch_verify_sampled(int logits_dtype, int B, int gamma, int V, const void* logits, const float* scores,
                                 const int* spine, const Sampling& smp, int* accept_len,
                                 int* bonus, void* scratch, int n_chunks, int chunk, int* status, hipStream_t st);
// G (fp32, optional copy G_out) and its bf16 hi/lo split planes Ghi, Glo = Ghi + M*H.
// Also zeroes n_clear uint64 words at `clear` (the persistent AR head's step tags).
hipError_t launch_gather_branch(int B, int gamma, int H, const float* reps,
                                const int* accept_len, float* G, float* G_out, bf16_t* Ghi,
                                uint64_t* clear, int64_t n_clear, int* status, hipStream_t st,
                                int* flag = nullptr);  // flag: set to 0 (the pruned head's fallback flag)
int ar_head_chunk(int dtype, int rank);  // vocabulary rows per AR-step workgroup
// Persistent bf16 AR head: grid size for (rank, V), 0 if unsupported; the partial buffer is
// [2][16][grid][2] uint64 and must hold zero tags when the launch starts.  Returns
// hipErrorNotSupported (nothing launched) when the configuration or the device's occupancy
// does not allow it.
int ar_persistent_grid(int rank, int V);
hipError_t launch_ar_head_persistent(int B, int gamma, int V, int rank, const float* logits, const void* E,
                                     const void* W, const int* bonus, int* drafts, int* next_spine, float* margins,
                                     uint64_t* part, int part_grid, int* status, const int* only_if,
                                     hipStream_t st, const Sampling& smp = Sampling{});
// bf16 with ppart (zero tags, ppart_grid = ar_persistent_grid) runs the persistent head when
// the device allows it; otherwise gamma+1 step kernels with partials in `part`.  With a
// non-NULL only_if, every kernel returns at once unless *only_if != 0 when it runs.
hipError_t launch_ar_head(int dtype, int B, int gamma, int V, int rank, const float* logits,
                          const void* E, const void* W, const int* bonus, int* drafts,
                          int* next_spine, float* margins, uint64_t* part, int n_chunks,
                          int chunk, uint64_t* ppart, int ppart_grid, int* status, const int* only_if,
                          hipStream_t st, const Sampling& smp = Sampling{});
// Exact bound-pruned head (head_prune.hip): top candidates per logit row, the largest W row
// norm, then all gamma steps over the candidates only.  Where a row or a step cannot be
// decided exactly it sets *flag != 0 (the flag is cleared first), and the caller runs
// launch_ar_head with only_if = flag, which recomputes every request.  `cand` holds
// head_prune_cand_bytes(B * gamma, V) bytes, `wpart` head_prune_wparts() floats.
// Returns hipErrorNotSupported (nothing launched) outside head_prune_supported().
bool head_prune_supported(int dtype, int gamma, int V, int rank);
int head_prune_splits(int rows, int V);
int head_prune_wparts();
size_t head_prune_cand_bytes(int rows, int V);
hipError_t launch_head_pruned(int dtype, int B, int gamma, int V, int rank, const float* logits, const void* E,
                              const void* W, const int* bonus, int* drafts, int* next_spine, float* margins,
                              uint64_t* cand, float* wpart, int* flag, int* status, hipStream_t st,
                              float inv_t = 1.0f, const float* wnorm_pre = nullptr, bool flag_cleared = false);
// max_v |W_v|^2 into out (one float); parts: head_prune_wparts() floats of scratch, scratch_flag
// one int.
hipError_t launch_head_prepare(int dtype, int rank, const void* W, int V, float* parts, int* scratch_flag, float* out,
                               hipStream_t st);
// Sampled head through the pruned steps: P = l * inv_t + Gumbel(key; head tag, b, i, v) for
// every head row (row b * gamma + i - 1), ranked by launch_head_pruned(..., P, inv_t); then,
// where the pruned steps decided every step (*flag == 0), the draft scores
// s_i = (l_i + W E(y_{i-1})) * inv_t of every vocabulary entry from the drafts now known, as a
// GEMM over the gathered E rows (`rows`: B * gamma * rank elements of the drafter dtype;
// `cbuf`: B * gamma * V floats of scratch; `ok`: one int of scratch).
hipError_t launch_perturb_logits(int B, int gamma, int V, const float* logits, float* P, const Sampling& smp,
                                 hipStream_t st);
hipError_t launch_draft_scores(int dtype, int B, int gamma, int V, int rank, const float* logits, const void* E,
                               const void* W, const int* bonus, const int* drafts, const Sampling& smp,
                               const int* flag, void* rows, float* cbuf, int* ok, hipStream_t st);
// Candidates of every branch row, off the serial path (bf16): reps [B, gamma+1, gamma, H]
// fp32 -> `cand` (head_cand_bytes: a 4 KB header with an overflow flag at 0 and the
// |W_v|^2 maxima at byte 256, then kTopK+1 keys per row); `split` holds 2 * rows * H bf16,
// `part` head_cand_part_bytes, `scratch` head_cand_scratch_bytes (8-byte aligned).  The top
// lists come from the hi plane of each row; their candidates are then rescored exactly and
// the bound widened by the lo plane's and the rounding's share.  emax2_pre: max_v |embed_v|^2 (one float, device) as
// launch_embed_prepare writes it, or NULL (one pass over the embedding per call).  The serial
// step then takes the accepted branch's rows.
size_t head_cand_bytes(int B, int gamma);
size_t head_cand_part_bytes(int B, int gamma, int V);
size_t head_cand_scratch_bytes(int B, int gamma);
hipError_t launch_branch_candidates(int B, int gamma, int H, int V, int rank, const float* reps, const void* embed,
                                    const void* W, const float* emax2_pre, void* cand, bf16_t* split, uint64_t* part,
                                    void* scratch, hipStream_t st);
// The greedy head's steps for B requests from candidates of their gathered rows G [B, gamma,
// H] fp32 (the same ranking and exact rescoring as above over B * gamma rows, `cand` of
// head_row_cand_bytes(B * gamma) bytes, split / part / scratch sized for at least those rows):
// drafts, next_spine and margins as the pruned head writes them, `flag` nonzero if some step
// is not proven (the caller then runs the full head).  wnorm_pre: the prepared max |W_v|^2, or
// NULL (one pass over W).
size_t head_row_cand_bytes(int rows);
hipError_t launch_head_ranked(int B, int gamma, int H, int V, int rank, const float* G, const void* embed,
                              const void* E, const void* W, const float* emax2_pre, const float* wnorm_pre,
                              const int* bonus, int* drafts, int* next_spine, float* margins, int* flag, int* status,
                              void* cand, bf16_t* split, uint64_t* part, void* scratch, hipStream_t st);
// max_v |embed_v|^2 of a [V, H] bf16 matrix into out (one float); parts: 512 floats of scratch.
hipError_t launch_embed_prepare(const void* embed, int V, int H, float* parts, float* out, hipStream_t st);
hipError_t launch_head_from_candidates(int B, int gamma, int V, int rank, const void* cand, const void* E,
                                       const void* W, const int* accept_len, const int* bonus, int* drafts,
                                       int* next_spine, float* margins, int* flag, int* status, hipStream_t st);

}  // namespace dpara
