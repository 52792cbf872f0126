/*
 * dpara.h - C ABI of the DPara drafter hot path on MI355X (gfx950).
 *
 * Method: "When Parallel Drafter Meets Parallel Speculative Decoding" (DPara).
 * One steady-state round (Algorithm 1) is:
 *   dpara_ctx_append               C <- [C, C_new]           (Section 3.3; Appendix D,
 *                                                              incremental projection)
 *   dpara_backbone_all_boundaries  Precompute: all d+1 acceptance boundaries in one
 *                                  forward under the tree mask (Section 3.2)
 *   dpara_verify_greedy            Verify verdict (r, b) from target logits (Section 2.1)
 *   dpara_select_and_head          select branch r, AR head y_i = argmax(l_i + W E(y_{i-1})),
 *                                  y_0 = b; next block (b, y_1..y_d) (Algorithm 1; the head
 *                                  equation of Section 3.2)
 * Around it:
 *   dpara_branch_candidates, dpara_select_and_head_cand   the head with every branch's base
 *                                  logits scored off the serial path (Algorithm 1, Precompute)
 *   dpara_verify_sampled, dpara_select_and_head_sampled   the sampling variant: speculative-
 *                                  sampling acceptance and y_i ~ softmax(z_i / T) (Section 2.1)
 *   dpara_target_forward[_hidden]  a verifying target on the same GPU (Section 4.3.2), also
 *                                  emitting the hidden states the drafter fuses
 *   dpara_fuse_features            C_new = RMSNorm(fc [h_1; ...; h_n]) (Section 3.2)
 * "d" in the paper is `gamma` here (draft length; gamma+1 boundaries).
 *
 * Conventions shared by every call:
 *  - Every pointer marked (device) is device memory owned by the caller.  The library
 *    never allocates or frees memory; scratch space is the caller's workspace `ws`.
 *  - Calls are asynchronous on the caller's HIP stream (`stream` is a hipStream_t; NULL
 *    means the default stream).  Nothing is read back to the host.
 *  - Return value: DPARA_OK or a negative DPARA_E_* code; dpara_last_error() then holds a
 *    message (thread-local).  Host-detected errors launch nothing.
 *  - Data errors only the device can see (token id outside [0, vocab), accepted length
 *    outside [0, gamma], context capacity exceeded) set bits in the int32 status word at
 *    byte offset 0 of the workspace (DPARA_STATUS_*); the offending item is clamped so
 *    no access leaves its buffer.  The library never clears the word itself:
 *    dpara_clear_status() enqueues a clear.
 *  - Matrices follow the Linear orientation [out, in]: y = x W^T.  Row-major throughout.
 *  - dtype (DPARA_F32 or DPARA_BF16) applies to matrices, embeddings, context features
 *    and the K/V cache; norm gains are always float32; the residual stream, the
 *    representations, logits and softmax are float32 in both modes.
 *  - Calls on one workspace must not overlap (same stream, or ordered by events), with one
 *    exception: a verification (dpara_verify_greedy or dpara_verify_sampled) may run on
 *    another stream beside dpara_ctx_append and dpara_backbone_all_boundaries.
 */
#ifndef DPARA_H
#define DPARA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  DPARA_OK = 0,
  DPARA_E_INVALID = -1,     /* null or misaligned pointer, bad shape, unsupported size */
  DPARA_E_UNSUPPORTED = -2, /* dtype / device architecture not supported */
  DPARA_E_WORKSPACE = -3,   /* ws_bytes smaller than dpara_workspace_bytes() */
  DPARA_E_CAPACITY = -4,    /* batch larger than the context cache's batch capacity */
  DPARA_E_HIP = -5          /* a HIP launch or runtime call failed */
};

enum { DPARA_F32 = 0, DPARA_BF16 = 1 };

enum {
  DPARA_STATUS_TOKEN_RANGE = 1,  /* a token id was outside [0, vocab) */
  DPARA_STATUS_CTX_FULL = 2,     /* an append would exceed ctx_cap; rows beyond it dropped */
  DPARA_STATUS_VERDICT_RANGE = 4, /* accept_len outside [0, gamma] */
  DPARA_STATUS_COUNT_RANGE = 8,   /* an append count n_new outside [0, n_max] (clamped) */
  DPARA_STATUS_HEAD_TIMEOUT = 16  /* the single-launch AR head's workgroups were not all resident
                                     together (e.g. the GPU was shared); its drafts are invalid */
};

/* Drafter shape.  Constraints: gamma in [1, 63]; head_dim in {64, 128};
 * n_q_heads % n_kv_heads == 0; hidden, ffn, n_q_heads*head_dim and ar_rank multiples
 * of 64; vocab >= 2.  qk_norm: per-head RMSNorm of q and k before RoPE (Qwen3). */
typedef struct dpara_config {
  int32_t n_layers;
  int32_t hidden;
  int32_t n_q_heads;
  int32_t n_kv_heads;
  int32_t head_dim;
  int32_t ffn;
  int32_t vocab;
  int32_t gamma;
  int32_t ar_rank;
  int32_t qk_norm;
  int32_t dtype;
  float rms_eps;
  float rope_base;
} dpara_config_t;

/* One pre-norm drafter block (device pointers; matrices in cfg dtype). */
typedef struct dpara_layer_weights {
  const float* attn_norm; /* [hidden] */
  const void* wq;         /* [n_q_heads*head_dim, hidden] */
  const void* wk;         /* [n_kv_heads*head_dim, hidden] */
  const void* wv;         /* [n_kv_heads*head_dim, hidden] */
  const float* q_norm;    /* [head_dim]; unused when qk_norm == 0 */
  const float* k_norm;    /* [head_dim]; unused when qk_norm == 0 */
  const void* wo;         /* [hidden, n_q_heads*head_dim] */
  const float* mlp_norm;  /* [hidden] */
  const void* w_gate;     /* [ffn, hidden] */
  const void* w_up;       /* [ffn, hidden] */
  const void* w_down;     /* [hidden, ffn] */
} dpara_layer_weights_t;

/* Frozen drafter parts (Section 3.2, "Trainable and frozen parameters"): the token
 * embedding doubles as the full-vocabulary LM head (tied); the AR head's low-rank token
 * embedding E and its vocabulary projection W (head equation, Section 3.2). */
typedef struct dpara_weights {
  const void* embed;                   /* [vocab, hidden] (device) */
  const void* mask_emb;                /* [hidden] (device): the mask-token input row */
  const float* final_norm;             /* [hidden] (device) */
  const void* ar_E;                    /* [vocab, ar_rank] (device) */
  const void* ar_W;                    /* [vocab, ar_rank] (device) */
  const dpara_layer_weights_t* layers; /* [n_layers] (HOST array of device pointers) */
  const float* ar_w_norm2_max;         /* optional (device, one float): max_v |ar_W[v]|^2 as
                                          dpara_head_prepare writes it; NULL: every head call
                                          computes it (one pass over ar_W) */
  const float* embed_norm2_max;        /* optional (device, one float): max_v |embed[v]|^2 as
                                          dpara_candidates_prepare writes it; NULL: every
                                          dpara_branch_candidates call computes it (one pass
                                          over embed) */
} dpara_weights_t;

/* Feature cache C kept as per-layer context K/V (Section 3.3: C over the accepted
 * history; Appendix D: incremental projection of cached history features).
 *   k: [n_layers, batch_cap, n_kv_heads, ctx_cap, head_dim]   (device, cfg dtype)
 *   v: [n_layers, batch_cap, n_kv_heads, head_dim, ctx_cap]   (device, cfg dtype; the
 *      value cache is stored transposed, positions contiguous)
 *   ctx_len: [batch_cap] int32 (device): cached positions per request.
 * Request b of a call uses slot b.  Positions are 0..ctx_len[b]-1. */
typedef struct dpara_ctx {
  void* k;
  void* v;
  int32_t* ctx_len;
  int32_t batch_cap;
  int32_t ctx_cap;
} dpara_ctx_t;

/* Bytes of workspace every call below needs for `batch` requests and a cache of
 * `ctx_cap` positions (the same workspace serves all four calls).  0 on invalid input. */
size_t dpara_workspace_bytes(const dpara_config_t* cfg, int32_t batch, int32_t ctx_cap);

/* C <- [C, C_new] (Algorithm 1, cache update; Section 3.3).
 * feats: [batch, n_max, hidden] (device, cfg dtype): fused target features of the newly
 *        verified positions (t_0..t_r of the last round).
 * n_new: [batch] int32 (device): rows of feats to append per request (0..n_max).
 * For every layer: k = RoPE(kNorm(W_k f)), v = W_v f at positions ctx_len[b] + i, written
 * into the cache; then ctx_len[b] += n_new[b].  Rows past ctx_cap are dropped and set
 * DPARA_STATUS_CTX_FULL.  Any n_max >= 1 is accepted (long prefills are chunked). */
int dpara_ctx_append(const dpara_config_t* cfg, const dpara_weights_t* w, const dpara_ctx_t* ctx,
                     int32_t batch, const void* feats, const int32_t* n_new, int32_t n_max,
                     void* ws, size_t ws_bytes, void* stream);

/* Algorithm 1, Precompute: the M-DFlash backbone on the spine t_0..t_gamma for all
 * gamma+1 acceptance boundaries in one forward (Section 3.2, tree mask).
 * spine: [batch, gamma+1] int32 (device); t_0 is the previous bonus.
 * reps:  [batch, gamma+1, gamma, hidden] float32 (device, output): final-norm hidden state
 *        of branch r's mask i at reps[b][r][i-1]; branch r assumes t_1..t_r accepted.
 * Rows per request: gamma+1 spine rows (position ctx_len[b]+j) and (gamma+1)*gamma mask
 * rows (branch r, mask i at position ctx_len[b]+r+i).  Spine t_j sees t_0..t_j; branch r's
 * masks see t_0..t_r and each other; every row sees the whole cache. */
int dpara_backbone_all_boundaries(const dpara_config_t* cfg, const dpara_weights_t* w,
                                  const dpara_ctx_t* ctx, int32_t batch, const int32_t* spine,
                                  float* reps, void* ws, size_t ws_bytes, void* stream);

/* dpara_backbone_all_boundaries that also writes the residual stream of every block row after
 * every drafter layer, for checking the layers one at a time against a reference (each layer is
 * the pre-norm block of Section 3.2's backbone; the tree mask is the same).
 * resid: [n_layers, batch, (gamma+1)^2, hidden] float32 (device, output, 16-byte aligned):
 *        resid[l][b][m] is row m of request b after layer l (row layout as for spine and reps:
 *        spine t_j at row j, branch r's mask i at row gamma+1+r*gamma+i-1).
 * reps and every other argument as for dpara_backbone_all_boundaries; reps come out bit for bit
 * the same.  Costs one extra write of the rows per layer. */
int dpara_backbone_trace(const dpara_config_t* cfg, const dpara_weights_t* w, const dpara_ctx_t* ctx,
                         int32_t batch, const int32_t* spine, float* reps, float* resid, void* ws,
                         size_t ws_bytes, void* stream);

/* Greedy verification (Section 2.1; Algorithm 1, Verify).
 * target_logits: [batch, gamma+1, vocab] (device), logits_dtype DPARA_F32 or DPARA_BF16:
 *                row j scores the token after t_j.
 * g_j = argmax_v logits[b][j][v] (lowest index on ties); accept_len[b] = number of leading
 * drafts with t_i == g_{i-1}; bonus[b] = g_{accept_len}.  Outputs (device, int32):
 * accept_len [batch], bonus [batch], target_argmax [batch, gamma+1] (may be NULL).
 * Out-of-range draft ids in spine set DPARA_STATUS_TOKEN_RANGE (they never match). */
int dpara_verify_greedy(const dpara_config_t* cfg, int32_t batch, const void* target_logits,
                        int32_t logits_dtype, const int32_t* spine, int32_t* accept_len,
                        int32_t* bonus, int32_t* target_argmax, void* ws, size_t ws_bytes,
                        void* stream);

/* dpara_verify_greedy without a workspace, for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid hipMalloc).  Same
 * arguments, outputs and results as dpara_verify_greedy; the partial argmax keys live in a
 * static device array of the library (1 MiB per GPU, kept until the process ends) instead of
 * `ws`.  Limit: 256 + batch * (gamma+1) * ceil(vocab / 4096) * 8 bytes must fit in 1 MiB (the
 * Qwen3 vocabulary at gamma 16: batch <= 202); larger calls return DPARA_E_WORKSPACE before
 * launching anything.
 * status: (device, int32, may be NULL) DPARA_STATUS_* bits are OR-ed into it (the caller clears
 *         it); with NULL, out-of-range draft ids are not reported (they still never match).
 * Every call on one GPU shares that GPU's array: calls that overlap in time on one GPU (other
 * streams, other threads) race and must be ordered by the caller. */
int dpara_verify_greedy_noalloc(const dpara_config_t* cfg, int32_t batch, const void* target_logits,
                                int32_t logits_dtype, const int32_t* spine, int32_t* accept_len,
                                int32_t* bonus, int32_t* target_argmax, int32_t* status, void* stream);

/* Select + AR head (Algorithm 1 after the barrier; head equation of Section 3.2).
 * reps: [batch, gamma+1, gamma, hidden] float32 (device) from the backbone.
 * accept_len, bonus: [batch] int32 (device) from verification.
 * gathered: [batch, gamma, hidden] float32 (device, may be NULL): reps[b][accept_len[b]],
 *           copied bit for bit.
 * drafts: [batch, gamma] int32 (device): y_1..y_gamma with
 *         l_i = gathered_i . embed^T, z_i = l_i + ar_W ar_E[y_{i-1}], y_0 = bonus,
 *         y_i = argmax z_i (lowest index on ties).
 * next_spine: [batch, gamma+1] int32 (device): (bonus, y_1..y_gamma).
 * margins: [batch, gamma] float32 (device, may be NULL): top1 - top2 of z_i.
 * With ar_rank in {64, 128, 256}, vocab >= 64 and gamma <= 63 the steps first run exactly
 * over a few candidates per step: the 16 largest l_i and a bound from the largest
 * remaining logit plus max_v |ar_W[v]| |ar_E[y_{i-1}]| (Cauchy-Schwarz), which proves the
 * step's top two when both candidates exceed it.  If any step of any request is not
 * proven, the int32 at byte offset 4 of `ws` is left nonzero (diagnostic; 0 otherwise) and
 * the full head below recomputes every request; the results are the same either way.
 * A bf16 drafter with more than 128 gathered rows (batch * gamma) and w->embed_norm2_max set
 * (dpara_candidates_prepare) takes the candidates another way: the gathered rows are ranked
 * by their bf16 hi parts and 64 candidates a row are rescored exactly, as in
 * dpara_branch_candidates (same drafts, next spine and margins bit for bit whenever every
 * step is proven); the two-plane LM head then runs only as part of the fallback.
 * The full head: bf16 drafters with ar_rank in {64, 128, 256}, vocab <= 2^18 and
 * batch <= 16 run the gamma head steps in one launch that needs all of its workgroups
 * resident at once (one per CU); if the GPU is shared so that they cannot all run, the
 * launch gives up after about 0.3 s per step and sets DPARA_STATUS_HEAD_TIMEOUT.  The
 * drafts, next_spine and margins of that call are then not valid (a workgroup whose wait
 * timed out stops there, and the steps from that one on are not all computed): the caller
 * checks the status word and repeats the call.  The single launch returns at once, without waiting, whenever
 * every pruned step was proven, so the bit can only be set by a call that needed the full
 * head.  (The timeout is not turned into a second, per-step pass on the device: that
 * needs one launch per step on every call, about 17 launches at gamma 16, even when
 * nothing timed out.)  Other configurations launch one kernel per step. */
int dpara_select_and_head(const dpara_config_t* cfg, const dpara_weights_t* w, int32_t batch,
                          const float* reps, const int32_t* accept_len, const int32_t* bonus,
                          float* gathered, int32_t* drafts, int32_t* next_spine, float* margins,
                          void* ws, size_t ws_bytes, void* stream);

/* Sampling variant (Algorithm 1's head loop draws y_i ~ softmax(z_i); Section 2.1's
 * distribution-preserving rejection sampling; the sampling appendix: temperature 1.0 for
 * target and drafter, top-p 1.0).
 *
 * Random numbers: U(seed; tag, b, i, v) = (2k + 1) / 2^24, k = the top 23 bits of word 0 of
 * Philox4x32-10 (Salmon, Moraes, Dror and Shaw, SC 2011) with counter (v, i, b, tag) and key
 * (seed mod 2^32, seed div 2^32); b is the request's index in the call's batch.  Tags: 1 head
 * draws (i = step, v = vocabulary id), 2 acceptance tests (i = draft index, v = 0), 3 bonus
 * draws (i = 0, v = vocabulary id).  A draw from softmax(x) is argmax_v x_v - log(-log U_v)
 * (Gumbel-max).  Callers pass a fresh seed per round; reusing one repeats the draws.  With
 * seed_dev non-NULL (device, one uint64, 8-byte aligned) the seed is read from there when the
 * kernels run and `seed` is ignored: a captured graph then takes a fresh seed per replay from
 * whatever the caller writes there between replays.
 *
 * dpara_select_and_head_sampled: dpara_select_and_head with y_i drawn from softmax(z_i / T)
 * (tag 1, step i) instead of argmax z_i; margins are top1 - top2 of z_i / T plus the noise.
 * draft_scores: [batch, gamma, vocab] float32 (device, may be NULL): s_i = z_i / T, the
 * tempered scores each draft was drawn from (the input of dpara_verify_sampled in the next
 * round).  As in the greedy head, the steps first run exactly over candidates: the 16 largest
 * of l_i / T + G_i (the noise is known before the steps) against the bound
 * max_v |ar_W[v]| |ar_E[y_{i-1}]| / T; if every step is proven, draft_scores come from one GEMM
 * over the drafts now known, else the int32 at byte offset 4 of `ws` is left nonzero and the
 * full head (same launch rules as dpara_select_and_head) recomputes every request and writes
 * the scores; the draws are the same either way up to float32 rounding.
 *
 * dpara_verify_sampled: speculative-sampling verification of the block t_0..t_gamma.
 * target_logits: [batch, gamma+1, vocab] (device, logits_dtype DPARA_F32 or DPARA_BF16,
 *                finite), row j scores the token after t_j; p_j = softmax(row j / T).
 * draft_scores:  [batch, gamma, vocab] float32 (device, finite): row i-1 holds the scores s
 *                draft t_i was drawn from; q_i = softmax(s).
 * Draft t_i (i = 1..gamma) is accepted while U(seed; 2, b, i, 0) < p_{i-1}(t_i) / q_i(t_i)
 * (tested in log space); accept_len[b] = r = the number of leading accepted drafts.  The
 * bonus is drawn (tag 3) from max(0, p_r - q_{r+1}) renormalised when r < gamma (from p_r
 * should rounding leave that empty) and from p_gamma when every draft is accepted.
 * Outputs (device, int32): accept_len [batch], bonus [batch].  Out-of-range draft ids set
 * DPARA_STATUS_TOKEN_RANGE and are never accepted.  ws: a workspace of
 * dpara_workspace_bytes(cfg, batch, ctx_cap) bytes; the call uses a region of its own, so it
 * may run concurrently with dpara_backbone_all_boundaries on the same workspace.
 * Both calls: temperature must be positive and finite (else DPARA_E_INVALID). */
int dpara_select_and_head_sampled(const dpara_config_t* cfg, const dpara_weights_t* w, int32_t batch,
                                  const float* reps, const int32_t* accept_len, const int32_t* bonus,
                                  float* gathered, int32_t* drafts, int32_t* next_spine, float* margins,
                                  float temperature, uint64_t seed, const uint64_t* seed_dev,
                                  float* draft_scores, void* ws, size_t ws_bytes, void* stream);
int dpara_verify_sampled(const dpara_config_t* cfg, int32_t batch, const void* target_logits,
                         int32_t logits_dtype, const float* draft_scores, const int32_t* spine,
                         float temperature, uint64_t seed, const uint64_t* seed_dev,
                         int32_t* accept_len, int32_t* bonus, void* ws, size_t ws_bytes, void* stream);

/* Weight preparation for the bound-pruned head steps (the Cauchy-Schwarz bound of
 * dpara_select_and_head): writes max_v |ar_W[v]|^2 into norm2_max (device, one float).  The
 * value depends on the weights only; set w->ar_w_norm2_max to it and every later head call
 * skips its own pass over ar_W, with the same results.  ws: a workspace of
 * dpara_workspace_bytes(cfg, 1, 64) bytes or more (scratch). */
int dpara_head_prepare(const dpara_config_t* cfg, const dpara_weights_t* w, float* norm2_max, void* ws,
                       size_t ws_bytes, void* stream);

/* Head variant with every branch's base logits computed off the serial path (Algorithm 1
 * computes the base logits during Precompute).
 * dpara_branch_candidates, issued after the backbone (for instance on its stream, where it
 * overlaps verification), ranks every row reps[b][r][i-1] against embed (the tied LM head) by
 * the row's bf16 part hi = bf16(x) alone, keeps per row the 16 largest of those scores, then
 * rescores these 16 with the full float32 row (applied as bf16 hi + lo, bit for bit the value
 * the LM head of dpara_select_and_head computes) and bounds every other logit of the row by the
 * largest hi score left out (the largest remaining one or the third largest of any
 * 128-column tile) plus |embed|max (|lo| + 6 hidden 2^-24 (|hi| + |lo|)): the lo part's
 * share by Cauchy-Schwarz and the float32 rounding of both sums.  It also keeps
 * max_v |ar_W[v]|^2.
 * cand: device buffer of dpara_branch_candidates_bytes(cfg, batch) bytes, 256-byte aligned;
 *       its layout is private to the library.
 * dpara_select_and_head_cand takes the accepted branch's candidates and produces the same
 * outputs as dpara_select_and_head (same inputs, same meaning): the gather, then the gamma
 * exact candidate steps; the LM head over the gathered rows and the full head run only if
 * some step is not proven (the int32 at byte offset 4 of `ws` is then nonzero).
 * bf16 drafters with ar_rank in {64, 128, 256}, vocab >= 64 and gamma <= 63 only (else
 * DPARA_E_UNSUPPORTED).  ws: a workspace of
 * dpara_workspace_bytes(cfg, batch, ctx_cap) bytes with ctx_cap >= 64.
 * dpara_candidates_prepare writes max_v |embed[v]|^2 into embed_norm2_max (device, one
 * float): set w->embed_norm2_max to it and later dpara_branch_candidates calls skip their
 * own pass over embed, with the same results.  ws: dpara_workspace_bytes(cfg, 1, 64) bytes
 * or more (scratch). */
size_t dpara_branch_candidates_bytes(const dpara_config_t* cfg, int32_t batch);
int dpara_branch_candidates(const dpara_config_t* cfg, const dpara_weights_t* w, int32_t batch,
                            const float* reps, void* cand, void* ws, size_t ws_bytes, void* stream);
int dpara_select_and_head_cand(const dpara_config_t* cfg, const dpara_weights_t* w, int32_t batch,
                               const float* reps, const void* cand, const int32_t* accept_len,
                               const int32_t* bonus, float* gathered, int32_t* drafts,
                               int32_t* next_spine, float* margins, void* ws, size_t ws_bytes,
                               void* stream);
int dpara_candidates_prepare(const dpara_config_t* cfg, const dpara_weights_t* w, float* embed_norm2_max,
                             void* ws, size_t ws_bytes, void* stream);

/* Target verification forward, used for the single-GPU overlap of verification and drafting
 * (Algorithm 1, Verify; Section 4.3.2 and Appendix D: both passes on two streams of one GPU).
 * A causal Qwen3-shaped decoder (same layer structure and dpara_config_t fields as the drafter;
 * gamma+1 = block length; ar_rank ignored; bf16 only) forwards each request's block
 * t_0..t_gamma at positions ctx_len[b]+j over its own per-layer K/V cache `ctx` (stored as
 * dpara_ctx_t describes; the cache is read, not updated), then the final RMSNorm (rounded to
 * bf16) and the untied LM head.
 * block:  [batch, gamma+1] int32 (device).
 * logits: [batch, gamma+1, vocab] (device, output), logits_dtype DPARA_F32 or DPARA_BF16;
 *         row j scores the token after t_j (the input of dpara_verify_greedy).
 * ws: a workspace of dpara_target_workspace_bytes() bytes (separate from the drafter's, so
 *     both passes can run concurrently on different streams). */
typedef struct dpara_target_weights {
  const void* embed;                   /* [vocab, hidden] (device) */
  const void* lm_head;                 /* [vocab, hidden] (device), untied */
  const float* final_norm;             /* [hidden] (device) */
  const dpara_layer_weights_t* layers; /* [n_layers] (HOST array of device pointers) */
} dpara_target_weights_t;

size_t dpara_target_workspace_bytes(const dpara_config_t* cfg, int32_t batch, int32_t ctx_cap);
int dpara_target_forward(const dpara_config_t* cfg, const dpara_target_weights_t* w,
                         const dpara_ctx_t* ctx, int32_t batch, const int32_t* block, void* logits,
                         int32_t logits_dtype, void* ws, size_t ws_bytes, void* stream);
/* The same forward, also emitting the block rows' hidden states after n_feat layers (the
 * multi-layer target features the drafter fuses, Section 3.2; dpara_fuse_features):
 * feat_layers: [n_feat] int32 (HOST array), layer indices in [0, n_layers), n_feat in [0, 8];
 * hidden: [batch, gamma+1, n_feat, hidden] bf16 (device, output, 16-byte aligned): the
 *         residual stream of row t_j after layer feat_layers[i] at hidden[b][j][i]. */
int dpara_target_forward_hidden(const dpara_config_t* cfg, const dpara_target_weights_t* w,
                                const dpara_ctx_t* ctx, int32_t batch, const int32_t* block,
                                void* logits, int32_t logits_dtype, const int32_t* feat_layers,
                                int32_t n_feat, void* hidden, void* ws, size_t ws_bytes, void* stream);

/* Feature fusion, the step before the cache update (Section 3.2, trainable and frozen
 * parameters: a learned linear map of the target's hidden states from several layers, joined
 * end to end, followed by a normalisation).  For every row x of `hidden` (the target's hidden states at
 * n_feat layers, concatenated): f = RMSNorm(x fc^T) * norm (eps cfg->rms_eps), the fused
 * feature dpara_ctx_append takes.  The projection accumulates in float32; f is rounded to
 * the cfg dtype.
 * hidden: [n_rows, n_feat * hidden] (device, cfg dtype, 16-byte aligned).
 * feats:  [n_rows, hidden] (device, cfg dtype, output, 16-byte aligned).
 * ws: dpara_fuse_workspace_bytes(cfg, n_rows, n_feat) bytes, 256-byte aligned (its own
 *     scratch: it need not be the drafter's workspace).  n_feat in [1, 8]; any n_rows >= 1
 *     (rows are processed in passes of at most 4096). */
typedef struct dpara_fusion_weights {
  const void* fc;     /* [hidden, n_feat * hidden] (device, cfg dtype), no bias */
  const float* norm;  /* [hidden] (device) */
  int32_t n_feat;
} dpara_fusion_weights_t;

size_t dpara_fuse_workspace_bytes(const dpara_config_t* cfg, int32_t n_rows, int32_t n_feat);
int dpara_fuse_features(const dpara_config_t* cfg, const dpara_fusion_weights_t* fw, int32_t n_rows,
                        const void* hidden, void* feats, void* ws, size_t ws_bytes, void* stream);

/* Enqueue a clear of the status word at byte offset 0 of `ws` (a fill kernel). */
int dpara_clear_status(void* ws, void* stream);

/* Per-phase tracing with HIP events recorded on the launching stream (off by default).
 * dpara_profile_enable(1) clears earlier records and starts recording a start/end event
 * pair around every kernel launch of a phase; dpara_profile_enable(0) stops.
 * dpara_profile_read(phase, &total_ms, &count) waits for the recorded events of `phase`
 * and returns their summed duration and launch count.  Phases: "append_gemm",
 * "append_store", "assemble", "rmsnorm", "qkv_gemm", "qk_norm_rope", "attn_ctx",
 * "attn_merge", "o_gemm", "gateup_gemm", "down_gemm", "final_norm", "verify", "gather",
 * "lm_head", "ar_step", "fuse_gemm", "fuse_norm".  Not for use while a stream is being captured into a graph. */
int dpara_profile_enable(int32_t on);
int dpara_profile_read(const char* phase, double* total_ms, int64_t* count);

/* Message for the last non-OK return on this thread ("" if none). */
const char* dpara_last_error(void);

/* ABI version: 100 * major + minor. */
int32_t dpara_version(void);

#ifdef __cplusplus
}
#endif
#endif /* DPARA_H */
