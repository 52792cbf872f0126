// C ABI of the DPara drafter hot path: argument validation, workspace planning and the
// launch sequence of each call on the caller's stream.  No allocation, no host sync.
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <cmath>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/dpara.h"
#include "internal.h"

#ifndef DPARA_ATTN_TARGET_WG
#define DPARA_ATTN_TARGET_WG 256
#endif

using namespace dpara;

namespace {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

int hip_fail(hipError_t e, const char* what) {
  return fail(DPARA_E_HIP, "%s: %s", what, hipGetErrorString(e));
}

#define HIP_TRY(expr, what)                    \
  do {                                         \
    hipError_t e_ = (expr);                    \
    if (e_ != hipSuccess) return hip_fail(e_, what); \
  } while (0)

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

size_t up256(size_t x) { return (x + 255) & ~(size_t)255; }

int check_cfg(const dpara_config_t* c) {
  if (!c) return fail(DPARA_E_INVALID, "cfg is NULL");
  if (c->n_layers < 1) return fail(DPARA_E_INVALID, "n_layers must be >= 1");
  if (c->hidden < 64 || c->hidden % 64) return fail(DPARA_E_INVALID, "hidden must be a positive multiple of 64");
  if (c->n_q_heads < 1 || c->n_kv_heads < 1 || c->n_q_heads % c->n_kv_heads)
    return fail(DPARA_E_INVALID, "n_q_heads must be a positive multiple of n_kv_heads");
  if (c->head_dim != 64 && c->head_dim != 128) return fail(DPARA_E_INVALID, "head_dim must be 64 or 128");
  if (c->ffn < 64 || c->ffn % 64) return fail(DPARA_E_INVALID, "ffn must be a positive multiple of 64");
  if (c->vocab < 2) return fail(DPARA_E_INVALID, "vocab must be >= 2");
  if (c->gamma < 1 || c->gamma > 63) return fail(DPARA_E_INVALID, "gamma must be in [1, 63]");
  if (c->ar_rank < 64 || c->ar_rank % 64 || c->ar_rank > 1024)
    return fail(DPARA_E_INVALID, "ar_rank must be a multiple of 64 in [64, 1024]");
  if (c->qk_norm != 0 && c->qk_norm != 1) return fail(DPARA_E_INVALID, "qk_norm must be 0 or 1");
  if (c->dtype != DPARA_F32 && c->dtype != DPARA_BF16) return fail(DPARA_E_UNSUPPORTED, "dtype must be F32 or BF16");
  if (!(c->rms_eps >= 0.f) || !(c->rope_base > 1.f)) return fail(DPARA_E_INVALID, "rms_eps >= 0 and rope_base > 1 required");
  return DPARA_OK;
}

#define CHECK_PTR(p, name)                                                         \
  do {                                                                             \
    if (!(p)) return fail(DPARA_E_INVALID, "%s is NULL", name);                    \
    if (!aligned16(p)) return fail(DPARA_E_INVALID, "%s is not 16-byte aligned", name); \
  } while (0)

int check_weights(const dpara_config_t* c, const dpara_weights_t* w, bool need_layers) {
  if (!w) return fail(DPARA_E_INVALID, "weights is NULL");
  CHECK_PTR(w->embed, "embed");
  if (need_layers) {
    CHECK_PTR(w->mask_emb, "mask_emb");
    CHECK_PTR(w->final_norm, "final_norm");
    if (!w->layers) return fail(DPARA_E_INVALID, "layers is NULL");
    for (int l = 0; l < c->n_layers; ++l) {
      const dpara_layer_weights_t& L = w->layers[l];
      CHECK_PTR(L.attn_norm, "attn_norm");
      CHECK_PTR(L.wq, "wq");
      CHECK_PTR(L.wk, "wk");
      CHECK_PTR(L.wv, "wv");
      CHECK_PTR(L.wo, "wo");
      CHECK_PTR(L.mlp_norm, "mlp_norm");
      CHECK_PTR(L.w_gate, "w_gate");
      CHECK_PTR(L.w_up, "w_up");
      CHECK_PTR(L.w_down, "w_down");
      if (c->qk_norm) {
        CHECK_PTR(L.q_norm, "q_norm");
        CHECK_PTR(L.k_norm, "k_norm");
      }
    }
  } else {
    CHECK_PTR(w->ar_E, "ar_E");
    CHECK_PTR(w->ar_W, "ar_W");
  }
  return DPARA_OK;
}

int check_ctx(const dpara_ctx_t* x, int batch) {
  if (!x) return fail(DPARA_E_INVALID, "ctx is NULL");
  CHECK_PTR(x->k, "ctx.k");
  CHECK_PTR(x->v, "ctx.v");
  if (!x->ctx_len) return fail(DPARA_E_INVALID, "ctx.ctx_len is NULL");
  if (x->ctx_cap < 64 || x->ctx_cap % 64) return fail(DPARA_E_INVALID, "ctx_cap must be a positive multiple of 64");
  if (batch > x->batch_cap) return fail(DPARA_E_CAPACITY, "batch %d exceeds ctx batch_cap %d", batch, x->batch_cap);
  return DPARA_OK;
}

// Workspace layout (byte offsets), shared by all calls.
struct Plan {
  int B, R, Rp, M, S, chunk, CH, esz;
  int s_qkv, s_o, s_down;  // split-K planes of the QKV, O and down projections
  bool afrag;              // normed activations in MFMA fragment order (QKV and gate/up GEMMs)
  bool qkv_fused;          // the QKV GEMM applies q/k-norm and RoPE in its epilogue
  int v_chunk, v_chunks, h_chunk, h_chunks;
  size_t X, A, QKV, Q, Kb, Vb, Opart, ML, O, Hmid, P, rope, vpart, G, Gsplit, logits, hpart, arpart, hcand, hwpart,
      hflag, F, KV32, rope_app, csplit, cpart, cscr, spart, plogits, erows;
  int ar_grid;  // persistent AR head grid (0: step kernels only)
  size_t total;
};

Plan make_plan(const dpara_config_t* c, int B, int ctx_cap, int R = 0) {
  Plan p{};
  p.B = B;
  p.R = R > 0 ? R : (c->gamma + 1) * (c->gamma + 1);
  p.Rp = (p.R + 63) / 64 * 64;
  p.M = B * p.R;
  p.esz = c->dtype == DPARA_BF16 ? 2 : 4;
  const int hd = c->head_dim, nq = c->n_q_heads, nkv = c->n_kv_heads, H = c->hidden;
  const int grp = nq / nkv;
  if (c->dtype == DPARA_BF16) {
    // Split each request's key blocks (context + in-block) over S workgroups so that the
    // MFMA pass launches at most about DPARA_ATTN_TARGET_WG workgroups (one per CU), with at
    // least 2 key blocks each; partial (O, m, l) traffic grows with S, so no more splits than
    // that.  Two workgroups fit on a CU, but more splits were measured slower at Qwen3-8B
    // batch 1 (targets 384 / 512 / 768: 44.9 / 43.2 / 50.7 us per layer with the fold, 41.8 at
    // 256).
    const int tiles = (grp * p.R + attn_rows_per_workgroup() - 1) / attn_rows_per_workgroup();
    const int base = B * nkv * tiles;
    const int max_blocks = (ctx_cap + 63) / 64 + p.Rp / 64;
    int S = DPARA_ATTN_TARGET_WG / base;
    const int max_s = min(max_blocks / 2, kMaxAttnSplits);
    if (S > max_s) S = max_s;
    if (S < 1) S = 1;
    if (base > DPARA_ATTN_TARGET_WG && max_s >= 2) {
      // Large batches: two workgroups fit on a CU (512 at once).  When the workgroups make at
      // most two rounds and the last one is at most 70% full, a split of two fills the rounds
      // (measured on MI355X at Qwen3-14B batch 8, context 8192: 1.5 -> 3 rounds, attention
      // 665 -> 609 us per layer with the fold); with more rounds, or contexts of mixed lengths,
      // the fold costs more than it saves (Qwen3-8B batch 16: 447 -> 479 us).
      constexpr int kSlots = 512;
      const int rounds = (base + kSlots - 1) / kSlots;
      if (rounds <= 2 && base % kSlots != 0 && base % kSlots <= kSlots * 7 / 10) S = 2;
    }
    p.S = S;
    p.chunk = 0;
  } else {
    p.S = 1;
    p.chunk = ctx_cap;
  }
  p.CH = p.R;
  p.v_chunk = 4096;
  p.v_chunks = (c->vocab + p.v_chunk - 1) / p.v_chunk;
  p.h_chunk = ar_head_chunk(c->dtype == DPARA_BF16 ? 1 : 0, c->ar_rank);
  p.h_chunks = (c->vocab + p.h_chunk - 1) / p.h_chunk;
  const int amode = c->dtype == DPARA_BF16 ? A_BF16 : A_F32;
  // From 65 to 320 rows the GEMMs fed by an RMSNorm read their activations in fragment order
  // (up to 64 rows the row-major LDS pipeline streams the weights faster: the 36-layer target
  // at batch 1, 5.2-5.4 -> 4.8 ms).
  p.afrag = c->dtype == DPARA_BF16 && p.M > 64 && p.M <= 320 && H % 256 == 0;
  p.s_qkv = gemm_splits(p.afrag ? A_BF16_FRAG : amode, EPI_STORE_F32, p.M, (nq + 2 * nkv) * hd, H);
  p.qkv_fused = c->dtype == DPARA_BF16 && hd == 128 && p.M > 1024 && p.s_qkv == 1;
  p.s_o = gemm_splits(amode, EPI_STORE_F32, p.M, H, nq * hd);
  p.s_down = gemm_splits(amode, EPI_STORE_F32, p.M, H, c->ffn);
  const size_t M = p.M;
  size_t off = 256;  // status header
  auto take = [&](size_t bytes) {
    size_t o = off;
    off += up256(bytes);
    return o;
  };
  // The verification regions come first: their offsets depend only on (cfg, B), never on
  // ctx_cap, so a verification may run beside the backbone on the same workspace.
  p.vpart = take((size_t)B * (c->gamma + 1) * p.v_chunks * 8);
  p.spart = take(verify_sampled_bytes(B, c->gamma, p.v_chunks));  // sampled verify: lse partials, bonus keys
  p.X = take(M * H * 4);
  p.A = take((p.afrag ? (M + 15) / 16 * 16 : M) * H * p.esz);
  p.QKV = take((size_t)p.s_qkv * M * (nq + 2 * nkv) * hd * 4);
  p.Q = take(M * (size_t)nq * hd * p.esz);
  p.Kb = take((size_t)B * nkv * p.Rp * hd * p.esz);  // [Rp][hd] per request and KV head
  p.Vb = take((size_t)B * nkv * hd * p.Rp * p.esz);  // transposed [hd][Rp] per request and KV head
  p.Opart = take((size_t)B * nq * p.R * p.S * hd * 4);
  p.ML = take((size_t)B * nq * p.R * p.S * 2 * 4);
  p.O = take(M * (size_t)nq * hd * p.esz);
  p.Hmid = take(M * (size_t)c->ffn * p.esz);
  p.P = take((size_t)(p.s_o > p.s_down ? p.s_o : p.s_down) * M * H * 4);  // O / down partial planes
  p.rope = take((size_t)B * (2 * c->gamma + 1) * (hd / 2) * 8);
  p.G = take((size_t)B * c->gamma * H * 4);
  p.Gsplit = take((size_t)2 * B * c->gamma * H * 2);  // bf16 hi and lo planes of G
  p.logits = take((size_t)B * c->gamma * c->vocab * 4);
  p.hpart = take((size_t)2 * B * p.h_chunks * 16);  // two step-parity slots
  p.ar_grid = (c->dtype == DPARA_BF16 && B <= 16) ? ar_persistent_grid(c->ar_rank, c->vocab) : 0;
  p.arpart = take((size_t)2 * 16 * p.ar_grid * 16);  // persistent head: [2][16][grid] x 2 words
  p.hcand = take(head_prune_cand_bytes(B * c->gamma, c->vocab));  // pruned head: candidate keys
  p.hwpart = take((size_t)head_prune_wparts() * 4);                // pruned head: |W_v|^2 maxima
  p.hflag = 4;  // pruned head: fallback flag, int32 in the header after the status word
  p.F = take((size_t)B * p.CH * H * p.esz);
  // append K|V planes of one layer group: split only when the append GEMM has at most 320
  // rows (16 planes max)
  const int app_layers = c->n_layers < kMaxAppendLayers ? c->n_layers : kMaxAppendLayers;
  const size_t kv_rows = (size_t)B * p.CH > 16 * 320 ? (size_t)B * p.CH : 16 * 320;
  p.KV32 = take(kv_rows * app_layers * 2 * nkv * hd * 4);
  p.rope_app = take((size_t)B * p.CH * (hd / 2) * 8);  // (cos, sin) of the appended rows' positions
  // branch candidates (bf16): hi/lo planes of every branch row and the per-tile top-2 words
  const size_t crows = (size_t)B * (c->gamma + 1) * c->gamma;
  p.csplit = take(c->dtype == DPARA_BF16 ? 2 * crows * H * 2 : 0);
  p.cpart = take(c->dtype == DPARA_BF16 ? head_cand_part_bytes(B, c->gamma, c->vocab) : 0);
  p.cscr = take(c->dtype == DPARA_BF16 ? head_cand_scratch_bytes(B, c->gamma) : 0);
  p.plogits = take((size_t)B * c->gamma * c->vocab * 4);  // sampled head: perturbed logits
  p.erows = take((size_t)B * c->gamma * c->ar_rank * p.esz);  // sampled head: E rows of the previous tokens
  p.total = off;
  return p;
}

std::mutex g_dev_mu;
int g_dev_ok[64];  // 0 unknown, 1 gfx950, -1 other

int check_device() {
  int dev = 0;
  HIP_TRY(hipGetDevice(&dev), "hipGetDevice");
  if (dev < 0 || dev >= 64) return fail(DPARA_E_UNSUPPORTED, "device index %d out of range", dev);
  std::lock_guard<std::mutex> lk(g_dev_mu);
  if (g_dev_ok[dev] == 0) {
    hipDeviceProp_t prop;
    HIP_TRY(hipGetDeviceProperties(&prop, dev), "hipGetDeviceProperties");
    g_dev_ok[dev] = strncmp(prop.gcnArchName, "gfx950", 6) == 0 ? 1 : -1;
  }
  if (g_dev_ok[dev] != 1) return fail(DPARA_E_UNSUPPORTED, "device %d is not gfx950 (MI355X)", dev);
  return DPARA_OK;
}

int check_ws(const Plan& p, void* ws, size_t ws_bytes) {
  if (!ws) return fail(DPARA_E_INVALID, "workspace is NULL");
  if (((uintptr_t)ws & 255u) != 0) return fail(DPARA_E_INVALID, "workspace must be 256-byte aligned");
  if (ws_bytes < p.total)
    return fail(DPARA_E_WORKSPACE, "workspace has %zu bytes, needs %zu", ws_bytes, p.total);
  return DPARA_OK;
}

template <typename T>
T* at(void* ws, size_t off) {
  return (T*)((char*)ws + off);
}

// ---------------------------------------------------------------- phase tracing
struct ProfRec {
  const char* phase;
  hipEvent_t a, b;
};
std::mutex g_prof_mu;
bool g_prof_on = false;
std::vector<ProfRec> g_prof;   // events are created once and reused across enables
size_t g_prof_used = 0;

}  // namespace

namespace dpara {
Phase::Phase(const char* name, hipStream_t s) : slot(-1), st(s) {
  if (!g_prof_on) return;
  std::lock_guard<std::mutex> lk(g_prof_mu);
  if (g_prof_used == g_prof.size()) {
    ProfRec r{name, nullptr, nullptr};
    if (hipEventCreate(&r.a) != hipSuccess || hipEventCreate(&r.b) != hipSuccess) return;
    g_prof.push_back(r);
  }
  slot = (int)g_prof_used++;
  g_prof[slot].phase = name;
  (void)hipEventRecord(g_prof[slot].a, st);
}
Phase::~Phase() {
  if (slot < 0) return;
  std::lock_guard<std::mutex> lk(g_prof_mu);
  (void)hipEventRecord(g_prof[slot].b, st);
}
}  // namespace dpara

namespace {
// Shared decoder pass over R block rows per request: row assembly, then every layer
// (RMSNorm -> QKV -> q/k-norm + RoPE -> attention over the cache and the in-block keys ->
// O + residual -> RMSNorm -> gate|up + SwiGLU -> down + residual).  spine_only selects the
// causal block (the target's verification pass); otherwise rows follow the tree layout.
// Leaves the residual stream in ws[p.X].
// hid_layers / n_hid / hid: optionally emit the rows' hidden state after those layers
// (hid[m * n_hid + j] after layer hid_layers[j], bf16).
// resid: optionally the float32 residual stream of every row after every layer
// (resid[l][m], [n_layers][M][H]).
int run_decoder(const dpara_config_t* cfg, const dpara_layer_weights_t* layers, const void* embed,
                const void* mask_emb, const dpara_ctx_t* ctx, int32_t batch, const int32_t* tokens,
                int spine_only, const Plan& p, void* ws, hipStream_t st, int* pending,
                const int32_t* hid_layers = nullptr, int n_hid = 0, void* hid = nullptr, float* resid = nullptr) {
  const int dt = cfg->dtype, H = cfg->hidden, hd = cfg->head_dim, nq = cfg->n_q_heads, nkv = cfg->n_kv_heads;
  const int g = cfg->gamma, R = p.R, M = p.M, F = cfg->ffn;
  const int amode = dt == DPARA_BF16 ? A_BF16 : A_F32;
  int* status = at<int>(ws, 0);
  float* X = at<float>(ws, p.X);
  const size_t layer_elems = (size_t)ctx->batch_cap * nkv * ctx->ctx_cap * hd;

  {
  Phase ph("assemble", st);
  HIP_TRY(launch_assemble_rows_rope(dt, batch, R, g, H, cfg->vocab, tokens, embed, mask_emb, X, status, 2 * g + 1,
                                    hd, cfg->rope_base, ctx->ctx_len, at<float2>(ws, p.rope), st),
          "assemble_rows");
  }
  float* P = at<float>(ws, p.P);
  int pend = 0;  // split-K planes of the last O / down projection not yet added into X
  for (int l = 0; l < cfg->n_layers; ++l) {
    const dpara_layer_weights_t& Lw = layers[l];
    {
    Phase ph("rmsnorm", st);
    if (p.afrag)
      HIP_TRY(launch_rmsnorm_frag(M, H, X, P, pend, (int64_t)M * H, Lw.attn_norm, cfg->rms_eps, at<void>(ws, p.A), st),
              "attn_norm");
    else
      HIP_TRY(launch_rmsnorm(dt, M, H, X, M, 0, 0, P, pend, (int64_t)M * H, 1, Lw.attn_norm, cfg->rms_eps,
                             at<void>(ws, p.A), st),
              "attn_norm");
    pend = 0;
    }
    GemmArgs q{};
    q.A = at<void>(ws, p.A);
    q.lda = H;
    q.B0 = Lw.wq;
    q.B1 = Lw.wk;
    q.B2 = Lw.wv;
    q.n1 = nq * hd;
    q.n2 = (nq + nkv) * hd;
    q.M = M;
    q.N = (nq + 2 * nkv) * hd;
    q.K = H;
    q.C = at<void>(ws, p.QKV);
    q.ldc = q.N;
    q.splits = p.s_qkv;
    if (p.qkv_fused) {
      // above 1024 rows (no split-K) the GEMM's epilogue applies q/k-norm and RoPE itself and
      // writes Q, K, V^T in bf16: the float32 Q|K|V never leaves the chip
      q.qkv.R = R;
      q.qkv.Rp = p.Rp;
      q.qkv.gamma = g;
      q.qkv.n_q = nq;
      q.qkv.n_kv = nkv;
      q.qkv.qk_norm = cfg->qk_norm;
      q.qkv.eps = cfg->rms_eps;
      q.qkv.qn = Lw.q_norm;
      q.qkv.kn = Lw.k_norm;
      q.qkv.table = at<float2>(ws, p.rope);
      q.qkv.Q = at<void>(ws, p.Q);
      q.qkv.Kb = at<void>(ws, p.Kb);
      q.qkv.Vb = at<void>(ws, p.Vb);
      Phase ph("qkv_gemm", st);
      HIP_TRY(launch_gemm(amode, EPI_QKV, q, st), "qkv gemm (fused q/k-norm and RoPE)");
    } else {
      {
      Phase ph("qkv_gemm", st);
      HIP_TRY(launch_gemm(p.afrag ? A_BF16_FRAG : amode, EPI_STORE_F32, q, st), "qkv gemm");
      }
      Phase ph("qk_norm_rope", st);
      HIP_TRY(launch_qk_norm_rope(dt, batch, R, p.Rp, g, nq, nkv, hd, cfg->qk_norm, cfg->rms_eps, at<float>(ws, p.QKV),
                                  p.s_qkv, Lw.q_norm, Lw.k_norm, at<float2>(ws, p.rope), at<void>(ws, p.Q),
                                  at<void>(ws, p.Kb), at<void>(ws, p.Vb), st),
              "qk_norm_rope");
    }
    AttnArgs aa{};
    aa.B = batch;
    aa.R = R;
    aa.gamma = g;
    aa.n_q = nq;
    aa.n_kv = nkv;
    aa.hd = hd;
    aa.Q = at<void>(ws, p.Q);
    aa.Kb = at<void>(ws, p.Kb);
    aa.Vb = at<void>(ws, p.Vb);
    aa.Rp = p.Rp;
    aa.Kc = (const char*)ctx->k + l * layer_elems * p.esz;
    aa.Vc = (const char*)ctx->v + l * layer_elems * p.esz;
    aa.cap = ctx->ctx_cap;
    aa.ctx_len = ctx->ctx_len;
    aa.S = p.S;
    aa.chunk = p.chunk;
    aa.Opart = at<float>(ws, p.Opart);
    aa.MLpart = at<float>(ws, p.ML);
    aa.O = at<void>(ws, p.O);
    aa.spine_only = spine_only;
    HIP_TRY(launch_attention(dt, aa, st), "attention");
    GemmArgs o{};
    o.A = at<void>(ws, p.O);
    o.lda = nq * hd;
    o.B0 = o.B1 = o.B2 = Lw.wo;
    o.n1 = o.n2 = H;
    o.M = M;
    o.N = H;
    o.K = nq * hd;
    o.C = P;
    o.ldc = H;
    o.splits = p.s_o;
    {
    Phase ph("o_gemm", st);
    HIP_TRY(launch_gemm(amode, EPI_STORE_F32, o, st), "o-proj gemm");
    }
    {
    Phase ph("rmsnorm", st);
    if (p.afrag)
      HIP_TRY(launch_rmsnorm_frag(M, H, X, P, p.s_o, (int64_t)M * H, Lw.mlp_norm, cfg->rms_eps, at<void>(ws, p.A), st),
              "mlp_norm");
    else
      HIP_TRY(launch_rmsnorm(dt, M, H, X, M, 0, 0, P, p.s_o, (int64_t)M * H, 1, Lw.mlp_norm, cfg->rms_eps,
                             at<void>(ws, p.A), st),
              "mlp_norm");
    }
    GemmArgs gu{};
    gu.A = at<void>(ws, p.A);
    gu.lda = H;
    gu.B0 = Lw.w_gate;
    gu.B1 = Lw.w_up;
    gu.B2 = Lw.w_up;
    gu.n1 = gu.n2 = F;
    gu.M = M;
    gu.N = F;
    gu.K = H;
    gu.C = at<void>(ws, p.Hmid);
    gu.ldc = F;
    {
    Phase ph("gateup_gemm", st);
    HIP_TRY(launch_gemm(p.afrag ? A_BF16_FRAG : amode, EPI_SWIGLU, gu, st), "gate/up gemm");
    }
    GemmArgs dn{};
    dn.A = at<void>(ws, p.Hmid);
    dn.lda = F;
    dn.B0 = dn.B1 = dn.B2 = Lw.w_down;
    dn.n1 = dn.n2 = H;
    dn.M = M;
    dn.N = H;
    dn.K = F;
    dn.C = P;
    dn.ldc = H;
    dn.splits = p.s_down;
    {
    Phase ph("down_gemm", st);
    HIP_TRY(launch_gemm(amode, EPI_STORE_F32, dn, st), "down gemm");
    }
    pend = p.s_down;
    for (int j = 0; j < n_hid; ++j)
      if (hid_layers[j] == l)
        HIP_TRY(launch_emit_hidden(M, H, X, P, pend, (int64_t)M * H, hid, n_hid, j, st), "emit hidden");
    if (resid)
      HIP_TRY(launch_emit_hidden(M, H, X, P, pend, (int64_t)M * H, resid + (size_t)l * M * H, 1, 0, st, 1),
              "emit residual");
  }
  *pending = pend;
  return DPARA_OK;
}

}  // namespace

// ---------------------------------------------------------------- allocation-free verification
// dpara_verify_greedy_noalloc takes its scratch from this array instead of a workspace: a
// 256-byte header (the status word when the caller passes none), then the per-chunk argmax
// partials of the verification.  Each GPU the library runs on holds its own copy until the
// process ends.  Host code uses only the address hipGetSymbolAddress returns for the current
// device, never the array's name.
constexpr size_t kNoAllocScratchBytes = (size_t)1 << 20;
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

namespace {
std::mutex g_scratch_mu;
void* g_scratch_dev[64];  // device address of `scratch` per device index (NULL until looked up)

// Device address of `scratch` on the current device, looked up once per device.
int scratch_address(void** out) {
  int dev = 0;
  HIP_TRY(hipGetDevice(&dev), "hipGetDevice");
  if (dev < 0 || dev >= 64) return fail(DPARA_E_UNSUPPORTED, "device index %d out of range", dev);
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_dev[dev]) {
    void* ptr = nullptr;
    HIP_TRY(hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)), "hipGetSymbolAddress(scratch)");
    if (!ptr) return fail(DPARA_E_HIP, "hipGetSymbolAddress(scratch) returned NULL");
    g_scratch_dev[dev] = ptr;
  }
  *out = g_scratch_dev[dev];
  return DPARA_OK;
}
}  // namespace

extern "C" {

int dpara_profile_enable(int32_t on) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  if (on) {
    for (size_t i = 0; i < g_prof_used; ++i) (void)hipEventSynchronize(g_prof[i].b);
    g_prof_used = 0;
  }
  g_prof_on = on != 0;
  return DPARA_OK;
}

int dpara_profile_read(const char* phase, double* total_ms, int64_t* count) {
  if (!phase || !total_ms || !count) return fail(DPARA_E_INVALID, "phase, total_ms and count must be non-NULL");
  std::lock_guard<std::mutex> lk(g_prof_mu);
  double t = 0.0;
  int64_t n = 0;
  for (size_t i = 0; i < g_prof_used; ++i) {
    if (strcmp(g_prof[i].phase, phase) != 0) continue;
    HIP_TRY(hipEventSynchronize(g_prof[i].b), "hipEventSynchronize");
    float ms = 0.f;
    HIP_TRY(hipEventElapsedTime(&ms, g_prof[i].a, g_prof[i].b), "hipEventElapsedTime");
    t += ms;
    ++n;
  }
  *total_ms = t;
  *count = n;
  return DPARA_OK;
}


int32_t dpara_version(void) { return 100; }

const char* dpara_last_error(void) { return g_err.c_str(); }

size_t dpara_workspace_bytes(const dpara_config_t* cfg, int32_t batch, int32_t ctx_cap) {
  if (check_cfg(cfg) != DPARA_OK || batch < 1 || ctx_cap < 64 || ctx_cap % 64) return 0;
  return make_plan(cfg, batch, ctx_cap).total;
}

int dpara_clear_status(void* ws, void* stream) {
  if (!ws) return fail(DPARA_E_INVALID, "workspace is NULL");
  int rc = check_device();
  if (rc) return rc;
  HIP_TRY(launch_clear_status((int*)ws, (hipStream_t)stream), "clear_status");
  return DPARA_OK;
}

int dpara_ctx_append(const dpara_config_t* cfg, const dpara_weights_t* w, const dpara_ctx_t* ctx, int32_t batch,
                     const void* feats, const int32_t* n_new, int32_t n_max, void* ws, size_t ws_bytes,
                     void* stream) {
  int rc = check_cfg(cfg);
  if (rc) return rc;
  if (batch < 1) return fail(DPARA_E_INVALID, "batch must be >= 1");
  if ((rc = check_ctx(ctx, batch))) return rc;
  if (!w || !w->layers) return fail(DPARA_E_INVALID, "weights or layers is NULL");
  for (int l = 0; l < cfg->n_layers; ++l) {
    CHECK_PTR(w->layers[l].wk, "wk");
    CHECK_PTR(w->layers[l].wv, "wv");
    if (cfg->qk_norm) CHECK_PTR(w->layers[l].k_norm, "k_norm");
  }
  CHECK_PTR(feats, "feats");
  if (!n_new) return fail(DPARA_E_INVALID, "n_new is NULL");
  if (n_max < 1) return fail(DPARA_E_INVALID, "n_max must be >= 1");
  const Plan p = make_plan(cfg, batch, ctx->ctx_cap);
  if ((rc = check_ws(p, ws, ws_bytes))) return rc;
  if ((rc = check_device())) return rc;

  hipStream_t st = (hipStream_t)stream;
  const int dt = cfg->dtype, H = cfg->hidden, hd = cfg->head_dim, nkv = cfg->n_kv_heads;
  int* status = at<int>(ws, 0);
  const size_t layer_elems = (size_t)ctx->batch_cap * nkv * ctx->ctx_cap * hd;
  const size_t esz = p.esz;
  const int CH = n_max < p.CH ? n_max : p.CH;  // rows per request per chunk
  for (int c0 = 0; c0 < n_max; c0 += CH) {
    HIP_TRY(launch_gather_feats(dt, batch, CH, c0, n_max, H, feats, at<void>(ws, p.F), st), "gather_feats");
    HIP_TRY(launch_rope_table(batch, CH, hd, cfg->rope_base, ctx->ctx_len, c0, at<float2>(ws, p.rope_app), st),
            "rope_table");
    // All layers project the same features: up to kMaxAppendLayers layers share one K|V GEMM
    // (weight segments W_k, W_v of each layer) and one store launch.
    for (int l0 = 0; l0 < cfg->n_layers; l0 += kMaxAppendLayers) {
      const int nl = cfg->n_layers - l0 < kMaxAppendLayers ? cfg->n_layers - l0 : kMaxAppendLayers;
      GemmArgs g{};
      g.A = at<void>(ws, p.F);
      g.lda = H;
      g.seg_rows = nkv * hd;
      KvLayers kn{};
      for (int j = 0; j < nl; ++j) {
        g.seg[2 * j] = w->layers[l0 + j].wk;
        g.seg[2 * j + 1] = w->layers[l0 + j].wv;
        kn.kn[j] = w->layers[l0 + j].k_norm;
      }
      g.M = batch * CH;
      g.N = nl * 2 * nkv * hd;
      g.K = H;
      g.C = at<void>(ws, p.KV32);
      g.ldc = g.N;
      g.splits = gemm_splits(dt == DPARA_BF16 ? A_BF16 : A_F32, EPI_STORE_F32, g.M, g.N, g.K);
      {
        Phase ph("append_gemm", st);
        HIP_TRY(launch_gemm(dt == DPARA_BF16 ? A_BF16 : A_F32, EPI_STORE_F32, g, st), "append kv gemm");
      }
      Phase ph("append_store", st);
      HIP_TRY(launch_kv_store(dt, batch, CH, c0, n_max, nkv, hd, cfg->qk_norm, cfg->rms_eps,
                              at<float2>(ws, p.rope_app), at<float>(ws, p.KV32), g.splits, nl, kn, n_new,
                              ctx->ctx_len, ctx->ctx_cap, (char*)ctx->k + l0 * layer_elems * esz,
                              (char*)ctx->v + l0 * layer_elems * esz, layer_elems, status, st),
              "kv_store");
    }
  }
  HIP_TRY(launch_ctx_len_update(batch, n_max, ctx->ctx_cap, n_new, ctx->ctx_len, status, st), "ctx_len_update");
  return DPARA_OK;
}

namespace {
int backbone_impl(const dpara_config_t* cfg, const dpara_weights_t* w, const dpara_ctx_t* ctx, int32_t batch,
                  const int32_t* spine, float* reps, float* resid, void* ws, size_t ws_bytes, void* stream) {
  int rc = check_cfg(cfg);
  if (rc) return rc;
  if (batch < 1) return fail(DPARA_E_INVALID, "batch must be >= 1");
  if ((rc = check_weights(cfg, w, true))) return rc;
  if ((rc = check_ctx(ctx, batch))) return rc;
  if (!spine) return fail(DPARA_E_INVALID, "spine is NULL");
  CHECK_PTR(reps, "reps");
  const Plan p = make_plan(cfg, batch, ctx->ctx_cap);
  if ((rc = check_ws(p, ws, ws_bytes))) return rc;
  if ((rc = check_device())) return rc;
  hipStream_t st = (hipStream_t)stream;
  int pend = 0;
  if ((rc = run_decoder(cfg, w->layers, w->embed, w->mask_emb, ctx, batch, spine, 0, p, ws, st, &pend, nullptr, 0,
                        nullptr, resid)))
    return rc;
  // reps[b][r][i-1] = final norm of mask rows: input row (m / nmask) * R + (g + 1 + m % nmask), with the
  // last down projection's split-K planes added
  const int g = cfg->gamma, R = p.R, H = cfg->hidden;
  const int nmask = R - g - 1;
  Phase ph("final_norm", st);
  HIP_TRY(launch_rmsnorm(0, batch * nmask, H, at<float>(ws, p.X), nmask, (int64_t)R * H, g + 1, at<float>(ws, p.P),
                         pend, (int64_t)p.M * H, 0, w->final_norm, cfg->rms_eps, reps, st),
          "final_norm");
  return DPARA_OK;
}
}  // namespace

int dpara_backbone_all_boundaries(const dpara_config_t* cfg, const dpara_weights_t* w, const dpara_ctx_t* ctx,
                                  int32_t batch, const int32_t* spine, float* reps, void* ws, size_t ws_bytes,
                                  void* stream) {
  return backbone_impl(cfg, w, ctx, batch, spine, reps, nullptr, ws, ws_bytes, stream);
}

int dpara_backbone_trace(const dpara_config_t* cfg, const dpara_weights_t* w, const dpara_ctx_t* ctx, int32_t batch,
                         const int32_t* spine, float* reps, float* resid, void* ws, size_t ws_bytes, void* stream) {
  CHECK_PTR(resid, "resid");
  return backbone_impl(cfg, w, ctx, batch, spine, reps, resid, ws, ws_bytes, stream);
}

size_t dpara_target_workspace_bytes(const dpara_config_t* cfg, int32_t batch, int32_t ctx_cap) {
  if (!cfg) return 0;
  dpara_config_t c = *cfg;
  c.ar_rank = 64;
  if (check_cfg(&c) != DPARA_OK || batch < 1 || ctx_cap < 64 || ctx_cap % 64) return 0;
  return make_plan(&c, batch, ctx_cap, cfg->gamma + 1).total;
}

int dpara_target_forward(const dpara_config_t* cfg, const dpara_target_weights_t* w, const dpara_ctx_t* ctx,
                         int32_t batch, const int32_t* block, void* logits, int32_t logits_dtype, void* ws,
                         size_t ws_bytes, void* stream) {
  return dpara_target_forward_hidden(cfg, w, ctx, batch, block, logits, logits_dtype, nullptr, 0, nullptr, ws,
                                     ws_bytes, stream);
}

int dpara_target_forward_hidden(const dpara_config_t* cfg, const dpara_target_weights_t* w, const dpara_ctx_t* ctx,
                                int32_t batch, const int32_t* block, void* logits, int32_t logits_dtype,
                                const int32_t* feat_layers, int32_t n_feat, void* hidden, void* ws,
                                size_t ws_bytes, void* stream) {
  if (!cfg) return fail(DPARA_E_INVALID, "cfg is NULL");
  if (n_feat < 0 || n_feat > 8) return fail(DPARA_E_INVALID, "n_feat must be in [0, 8]");
  if (n_feat > 0) {
    if (!feat_layers) return fail(DPARA_E_INVALID, "feat_layers is NULL");
    CHECK_PTR(hidden, "hidden");
    if (!aligned16(hidden)) return fail(DPARA_E_INVALID, "hidden is not 16-byte aligned");
    for (int j = 0; j < n_feat; ++j)
      if (feat_layers[j] < 0 || feat_layers[j] >= cfg->n_layers)
        return fail(DPARA_E_INVALID, "feat_layers[%d] = %d outside [0, n_layers)", j, feat_layers[j]);
  }
  dpara_config_t c = *cfg;
  c.ar_rank = 64;  // the target has no AR head
  int rc = check_cfg(&c);
  if (rc) return rc;
  if (batch < 1) return fail(DPARA_E_INVALID, "batch must be >= 1");
  if (c.dtype != DPARA_BF16) return fail(DPARA_E_UNSUPPORTED, "the target forward runs in bf16 only");
  if (logits_dtype != DPARA_F32 && logits_dtype != DPARA_BF16)
    return fail(DPARA_E_UNSUPPORTED, "logits_dtype must be F32 or BF16");
  if (!w || !w->layers) return fail(DPARA_E_INVALID, "target weights or layers is NULL");
  CHECK_PTR(w->embed, "embed");
  CHECK_PTR(w->lm_head, "lm_head");
  CHECK_PTR(w->final_norm, "final_norm");
  dpara_weights_t shim{};
  shim.embed = w->embed;
  shim.mask_emb = w->embed;
  shim.final_norm = w->final_norm;
  shim.layers = w->layers;
  if ((rc = check_weights(&c, &shim, true))) return rc;
  if ((rc = check_ctx(ctx, batch))) return rc;
  if (!block) return fail(DPARA_E_INVALID, "block is NULL");
  CHECK_PTR(logits, "logits");
  const Plan p = make_plan(&c, batch, ctx->ctx_cap, c.gamma + 1);
  if ((rc = check_ws(p, ws, ws_bytes))) return rc;
  if ((rc = check_device())) return rc;
  hipStream_t st = (hipStream_t)stream;
  int pend = 0;
  if ((rc = run_decoder(&c, w->layers, w->embed, w->embed, ctx, batch, block, 1, p, ws, st, &pend, feat_layers,
                        n_feat, hidden)))
    return rc;
  const int H = c.hidden, M = p.M;
  {
    Phase ph("final_norm", st);
    HIP_TRY(launch_rmsnorm(DPARA_BF16, M, H, at<float>(ws, p.X), M, 0, 0, at<float>(ws, p.P), pend, (int64_t)M * H,
                           0, w->final_norm, c.rms_eps, at<void>(ws, p.A), st),
            "target final norm");
  }
  GemmArgs lm{};
  lm.A = at<void>(ws, p.A);
  lm.lda = H;
  lm.B0 = lm.B1 = lm.B2 = w->lm_head;
  lm.n1 = lm.n2 = c.vocab;
  lm.M = M;
  lm.N = c.vocab;
  lm.K = H;
  lm.C = logits;
  lm.ldc = c.vocab;
  Phase ph("lm_head", st);
  HIP_TRY(launch_gemm(A_BF16, logits_dtype == DPARA_BF16 ? EPI_STORE_BF16 : EPI_STORE_F32, lm, st),
          "target lm head");
  return DPARA_OK;
}

int dpara_verify_greedy(const dpara_config_t* cfg, int32_t batch, const void* target_logits, int32_t logits_dtype,
                        const int32_t* spine, int32_t* accept_len, int32_t* bonus, int32_t* target_argmax,
                        void* ws, size_t ws_bytes, void* stream) {
  int rc = check_cfg(cfg);
  if (rc) return rc;
  if (batch < 1) return fail(DPARA_E_INVALID, "batch must be >= 1");
  if (logits_dtype != DPARA_F32 && logits_dtype != DPARA_BF16)
    return fail(DPARA_E_UNSUPPORTED, "logits_dtype must be F32 or BF16");
  if (!target_logits || !spine || !accept_len || !bonus)
    return fail(DPARA_E_INVALID, "target_logits, spine, accept_len and bonus must be non-NULL");
  const Plan p = make_plan(cfg, batch, 64);
  if (!ws) return fail(DPARA_E_INVALID, "workspace is NULL");
  const size_t need = p.vpart + up256((size_t)batch * (cfg->gamma + 1) * p.v_chunks * 8);
  if (ws_bytes < need) return fail(DPARA_E_WORKSPACE, "workspace has %zu bytes, needs %zu", ws_bytes, need);
  if ((rc = check_device())) return rc;
  HIP_TRY(launch_verify(logits_dtype, batch, cfg->gamma, cfg->vocab, target_logits, spine, accept_len, bonus,
                        target_argmax, at<uint64_t>(ws, p.vpart), p.v_chunks, p.v_chunk, at<int>(ws, 0),
                        (hipStream_t)stream),
          "verify");
  return DPARA_OK;
}

int dpara_verify_greedy_noalloc(const dpara_config_t* cfg, int32_t batch, const void* target_logits,
                                int32_t logits_dtype, const int32_t* spine, int32_t* accept_len, int32_t* bonus,
                                int32_t* target_argmax, int32_t* status, void* stream) {
  int rc = check_cfg(cfg);
  if (rc) return rc;
  if (batch < 1) return fail(DPARA_E_INVALID, "batch must be >= 1");
  if (logits_dtype != DPARA_F32 && logits_dtype != DPARA_BF16)
    return fail(DPARA_E_UNSUPPORTED, "logits_dtype must be F32 or BF16");
  if (!target_logits || !spine || !accept_len || !bonus)
    return fail(DPARA_E_INVALID, "target_logits, spine, accept_len and bonus must be non-NULL");
  if (status && ((uintptr_t)status & 3u)) return fail(DPARA_E_INVALID, "status is not 4-byte aligned");
  const Plan p = make_plan(cfg, batch, 64);
  const size_t need = 256 + up256((size_t)batch * (cfg->gamma + 1) * p.v_chunks * 8);
  if (need > kNoAllocScratchBytes)
    return fail(DPARA_E_WORKSPACE,
                "batch %d x %d rows x %d vocabulary chunks needs %zu bytes of scratch; the allocation-free "
                "verification holds %zu", batch, cfg->gamma + 1, p.v_chunks, need, kNoAllocScratchBytes);
  if ((rc = check_device())) return rc;
  void* sp = nullptr;
  if ((rc = scratch_address(&sp))) return rc;
  HIP_TRY(launch_verify(logits_dtype, batch, cfg->gamma, cfg->vocab, target_logits, spine, accept_len, bonus,
                        target_argmax, (uint64_t*)((char*)sp + 256), p.v_chunks, p.v_chunk,
                        status ? status : (int*)sp, (hipStream_t)stream),
          "verify (no allocation)");
  return DPARA_OK;
}

namespace {
// Gather, LM head, then the AR head: greedy (smp == nullptr: bound-pruned steps first, the
// full head only where a step is not proven) or sampled (the full head with Gumbel noise).
int select_and_head_impl(const dpara_config_t* cfg, const dpara_weights_t* w, int32_t batch, const float* reps,
                         const int32_t* accept_len, const int32_t* bonus, float* gathered, int32_t* drafts,
                         int32_t* next_spine, float* margins, void* ws, size_t ws_bytes, void* stream,
                         const Sampling* smp) {
  int rc = check_cfg(cfg);
  if (rc) return rc;
  if (batch < 1) return fail(DPARA_E_INVALID, "batch must be >= 1");
  if ((rc = check_weights(cfg, w, false))) return rc;
  CHECK_PTR(reps, "reps");
  if (gathered && !aligned16(gathered)) return fail(DPARA_E_INVALID, "gathered is not 16-byte aligned");
  if (!accept_len || !bonus || !drafts || !next_spine)
    return fail(DPARA_E_INVALID, "accept_len, bonus, drafts and next_spine must be non-NULL");
  const Plan p = make_plan(cfg, batch, 64);
  if (!ws) return fail(DPARA_E_INVALID, "workspace is NULL");
  if (((uintptr_t)ws & 255u) != 0) return fail(DPARA_E_INVALID, "workspace must be 256-byte aligned");
  size_t need = p.hwpart + up256((size_t)head_prune_wparts() * 4);
  if (smp)  // the sampled head also uses the perturbed-logit and E-row regions at the end
    need = p.erows + up256((size_t)batch * cfg->gamma * cfg->ar_rank * p.esz);
  if (ws_bytes < need) return fail(DPARA_E_WORKSPACE, "workspace has %zu bytes, needs %zu", ws_bytes, need);
  if ((rc = check_device())) return rc;

  hipStream_t st = (hipStream_t)stream;
  const int g = cfg->gamma, H = cfg->hidden, V = cfg->vocab;
  int* status = at<int>(ws, 0);
  float* G = at<float>(ws, p.G);
  bf16_t* Gs = at<bf16_t>(ws, p.Gsplit);
  // the gather also clears the pruned head's fallback flag (no kernel before the pruned
  // steps reads it)
  HIP_TRY(launch_gather_branch(batch, g, H, reps, accept_len, G, gathered, Gs, at<uint64_t>(ws, p.arpart),
                               (int64_t)2 * 16 * p.ar_grid * 2, status, st, at<int>(ws, p.hflag)),
          "gather_branch");
  const bool bf = cfg->dtype == DPARA_BF16;
  // Greedy bf16 head over more than 128 gathered rows with the embedding's max row norm
  // prepared: candidates from the rows' bf16 hi parts, rescored exactly (the branch-candidates
  // machinery over the gathered rows only), instead of the two-plane LM head and a top-k pass
  // over its float32 logits; the LM head then runs only if a step is not proven.  Same drafts,
  // next spine and margins bit for bit when every step is proven (the rescored logits are the
  // LM head's own).  Batch 16: the head 720 -> about 480 us.
  const bool ranked = bf && !smp && batch * g > 128 && w->embed_norm2_max && H % 64 == 0 &&
                      head_prune_supported(1, g, V, cfg->ar_rank) &&
                      ws_bytes >= p.plogits + up256(head_row_cand_bytes(batch * g));
  if (ranked) {
    int* hflag = at<int>(ws, p.hflag);
    HIP_TRY(launch_head_ranked(batch, g, H, V, cfg->ar_rank, G, w->embed, w->ar_E, w->ar_W, w->embed_norm2_max,
                               w->ar_w_norm2_max, bonus, drafts, next_spine, margins, hflag, status,
                               at<void>(ws, p.plogits), at<bf16_t>(ws, p.csplit), at<uint64_t>(ws, p.cpart),
                               at<void>(ws, p.cscr), st),
            "ranked head");
    GemmArgs lm{};
    lm.A = Gs;
    lm.lo_off = (int64_t)batch * g * H;
    lm.lda = H;
    lm.B0 = lm.B1 = lm.B2 = w->embed;
    lm.n1 = lm.n2 = V;
    lm.M = batch * g;
    lm.N = V;
    lm.K = H;
    lm.C = at<void>(ws, p.logits);
    lm.ldc = V;
    lm.only_if = hflag;  // only if some step was not proven
    {
      Phase ph("lm_head", st);
      HIP_TRY(launch_gemm(A_BF16_DUAL, EPI_STORE_F32, lm, st), "lm head gemm");
    }
    HIP_TRY(launch_ar_head(cfg->dtype, batch, g, V, cfg->ar_rank, at<float>(ws, p.logits), w->ar_E, w->ar_W, bonus,
                           drafts, next_spine, margins, at<uint64_t>(ws, p.hpart), p.h_chunks, p.h_chunk,
                           p.ar_grid ? at<uint64_t>(ws, p.arpart) : nullptr, p.ar_grid, status, hflag, st),
            "ar head");
    return DPARA_OK;
  }
  GemmArgs lm{};
  lm.A = bf ? (const void*)Gs : (const void*)G;
  lm.lo_off = (int64_t)batch * g * H;
  lm.lda = H;
  lm.B0 = lm.B1 = lm.B2 = w->embed;
  lm.n1 = lm.n2 = V;
  lm.M = batch * g;
  lm.N = V;
  lm.K = H;
  lm.C = at<void>(ws, p.logits);
  lm.ldc = V;
  {
    Phase ph("lm_head", st);
    HIP_TRY(launch_gemm(bf ? A_BF16_DUAL : A_F32, EPI_STORE_F32, lm, st), "lm head gemm");
  }
  if (smp) {
    // Exact bound-pruned steps over the perturbed logits first; the full sampled head runs only
    // if some step is not proven (it then writes the scores itself), else the scores kernel does.
    int* hflag = at<int>(ws, p.hflag);
    hipError_t pe = hipErrorNotSupported;
    if (head_prune_supported(cfg->dtype, g, V, cfg->ar_rank)) {
      HIP_TRY(launch_perturb_logits(batch, g, V, at<float>(ws, p.logits), at<float>(ws, p.plogits), *smp, st),
              "perturbed logits");
      pe = launch_head_pruned(cfg->dtype, batch, g, V, cfg->ar_rank, at<float>(ws, p.plogits), w->ar_E, w->ar_W,
                              bonus, drafts, next_spine, margins, at<uint64_t>(ws, p.hcand), at<float>(ws, p.hwpart),
                              hflag, status, st, smp->inv_t, w->ar_w_norm2_max, true);
      if (pe != hipSuccess && pe != hipErrorNotSupported) return hip_fail(pe, "sampled pruned head");
    }
    HIP_TRY(launch_ar_head(cfg->dtype, batch, g, V, cfg->ar_rank, at<float>(ws, p.logits), w->ar_E, w->ar_W, bonus,
                           drafts, next_spine, margins, at<uint64_t>(ws, p.hpart), p.h_chunks, p.h_chunk,
                           p.ar_grid ? at<uint64_t>(ws, p.arpart) : nullptr, p.ar_grid, status,
                           pe == hipSuccess ? hflag : nullptr, st, *smp),
            "sampled ar head");
    if (pe == hipSuccess && smp->scores)
      HIP_TRY(launch_draft_scores(cfg->dtype, batch, g, V, cfg->ar_rank, at<float>(ws, p.logits), w->ar_E, w->ar_W,
                                  bonus, drafts, *smp, hflag, at<void>(ws, p.erows), at<float>(ws, p.plogits),
                                  at<int>(ws, 8), st),
              "draft scores");
    return DPARA_OK;
  }
  // Exact bound-pruned steps first; the full head then runs only if some step could not be
  // decided from the candidates (its kernels return at once otherwise).
  int* hflag = at<int>(ws, p.hflag);
  const hipError_t pe = launch_head_pruned(cfg->dtype, batch, g, V, cfg->ar_rank, at<float>(ws, p.logits),
                                           w->ar_E, w->ar_W, bonus, drafts, next_spine, margins,
                                           at<uint64_t>(ws, p.hcand), at<float>(ws, p.hwpart), hflag, status, st,
                                           1.0f, w->ar_w_norm2_max, true);
  if (pe != hipSuccess && pe != hipErrorNotSupported) return hip_fail(pe, "pruned head");
  HIP_TRY(launch_ar_head(cfg->dtype, batch, g, V, cfg->ar_rank, at<float>(ws, p.logits), w->ar_E, w->ar_W, bonus,
                         drafts, next_spine, margins, at<uint64_t>(ws, p.hpart), p.h_chunks, p.h_chunk,
                         p.ar_grid ? at<uint64_t>(ws, p.arpart) : nullptr, p.ar_grid, status,
                         pe == hipSuccess ? hflag : nullptr, st),
          "ar head");
  return DPARA_OK;
}

}  // namespace

int dpara_head_prepare(const dpara_config_t* cfg, const dpara_weights_t* w, float* norm2_max, void* ws,
                       size_t ws_bytes, void* stream) {
  int rc = check_cfg(cfg);
  if (rc) return rc;
  if (!w || !w->ar_W) return fail(DPARA_E_INVALID, "weights or ar_W is NULL");
  CHECK_PTR(norm2_max, "norm2_max");
  if (!ws || ((uintptr_t)ws & 255u) != 0) return fail(DPARA_E_INVALID, "workspace is NULL or not 256-byte aligned");
  const Plan p = make_plan(cfg, 1, 64);
  const size_t need = p.hwpart + up256((size_t)head_prune_wparts() * 4);
  if (ws_bytes < need) return fail(DPARA_E_WORKSPACE, "workspace has %zu bytes, needs %zu", ws_bytes, need);
  if (cfg->ar_rank != 64 && cfg->ar_rank != 128 && cfg->ar_rank != 256)
    return fail(DPARA_E_UNSUPPORTED, "the pruned head needs ar_rank in {64, 128, 256}");
  if ((rc = check_device())) return rc;
  HIP_TRY(launch_head_prepare(cfg->dtype, cfg->ar_rank, w->ar_W, cfg->vocab, at<float>(ws, p.hwpart),
                              at<int>(ws, 12), norm2_max, (hipStream_t)stream),
          "head prepare");
  return DPARA_OK;
}

namespace {
// Temperature and seed of the sampling variant: the generator's key is the seed's two
// 32-bit halves.
int make_sampling(float temperature, uint64_t seed, const uint64_t* seed_dev, float* scores, Sampling* smp) {
  if (!(temperature > 0.f) || !std::isfinite(temperature) || !std::isfinite(1.0f / temperature))
    return fail(DPARA_E_INVALID, "temperature must be positive and finite, got %g", (double)temperature);
  if ((uintptr_t)seed_dev % 8 != 0) return fail(DPARA_E_INVALID, "seed_dev is not 8-byte aligned");
  smp->on = 1;
  smp->inv_t = 1.0f / temperature;
  smp->k0 = (uint32_t)(seed & 0xFFFFFFFFu);
  smp->k1 = (uint32_t)(seed >> 32);
  smp->seed_dev = seed_dev;
  smp->scores = scores;
  return DPARA_OK;
}
}  // namespace

int dpara_select_and_head(const dpara_config_t* cfg, const dpara_weights_t* w, int32_t batch, const float* reps,
                          const int32_t* accept_len, const int32_t* bonus, float* gathered, int32_t* drafts,
                          int32_t* next_spine, float* margins, void* ws, size_t ws_bytes, void* stream) {
  return select_and_head_impl(cfg, w, batch, reps, accept_len, bonus, gathered, drafts, next_spine, margins, ws,
                              ws_bytes, stream, nullptr);
}

int dpara_select_and_head_sampled(const dpara_config_t* cfg, const dpara_weights_t* w, int32_t batch,
                                  const float* reps, const int32_t* accept_len, const int32_t* bonus,
                                  float* gathered, int32_t* drafts, int32_t* next_spine, float* margins,
                                  float temperature, uint64_t seed, const uint64_t* seed_dev, float* draft_scores,
                                  void* ws, size_t ws_bytes, void* stream) {
  Sampling smp{};
  const int rc = make_sampling(temperature, seed, seed_dev, draft_scores, &smp);
  if (rc) return rc;
  return select_and_head_impl(cfg, w, batch, reps, accept_len, bonus, gathered, drafts, next_spine, margins, ws,
                              ws_bytes, stream, &smp);
}

int dpara_verify_sampled(const dpara_config_t* cfg, int32_t batch, const void* target_logits, int32_t logits_dtype,
                         const float* draft_scores, const int32_t* spine, float temperature, uint64_t seed,
                         const uint64_t* seed_dev, int32_t* accept_len, int32_t* bonus, void* ws, size_t ws_bytes,
                         void* stream) {
  int rc = check_cfg(cfg);
  if (rc) return rc;
  if (batch < 1) return fail(DPARA_E_INVALID, "batch must be >= 1");
  if (logits_dtype != DPARA_F32 && logits_dtype != DPARA_BF16)
    return fail(DPARA_E_UNSUPPORTED, "logits_dtype must be F32 or BF16");
  if (!target_logits || !draft_scores || !spine || !accept_len || !bonus)
    return fail(DPARA_E_INVALID, "target_logits, draft_scores, spine, accept_len and bonus must be non-NULL");
  Sampling smp{};
  if ((rc = make_sampling(temperature, seed, seed_dev, nullptr, &smp))) return rc;
  const Plan p = make_plan(cfg, batch, 64);
  if (!ws) return fail(DPARA_E_INVALID, "workspace is NULL");
  if (((uintptr_t)ws & 255u) != 0) return fail(DPARA_E_INVALID, "workspace must be 256-byte aligned");
  const size_t need = p.spart + verify_sampled_bytes(batch, cfg->gamma, p.v_chunks);
  if (ws_bytes < need) return fail(DPARA_E_WORKSPACE, "workspace has %zu bytes, needs %zu", ws_bytes, need);
  if ((rc = check_device())) return rc;
  HIP_TRY(launch_verify_sampled(logits_dtype, batch, cfg->gamma, cfg->vocab, target_logits, draft_scores, spine,
                                smp, accept_len, bonus, at<void>(ws, p.spart), p.v_chunks,
                                p.v_chunk, at<int>(ws, 0), (hipStream_t)stream),
          "sampled verify");
  return DPARA_OK;
}

// Feature fusion: passes of at most kFuseChunk rows; the fp32 projection goes to split-K
// planes (up to 16 of them for a pass of at most 320 rows) that the RMSNorm adds.
namespace {
constexpr int kFuseChunk = 4096;
size_t fuse_ws_bytes(const dpara_config_t* c, int n_rows) {
  const size_t small = (size_t)16 * (n_rows < 320 ? n_rows : 320);
  const size_t big = (size_t)(n_rows < kFuseChunk ? n_rows : kFuseChunk);
  return 256 + up256((small > big ? small : big) * c->hidden * 4);
}
}  // namespace

size_t dpara_fuse_workspace_bytes(const dpara_config_t* cfg, int32_t n_rows, int32_t n_feat) {
  if (check_cfg(cfg) || n_rows < 1 || n_feat < 1 || n_feat > 8) return 0;
  return fuse_ws_bytes(cfg, n_rows);
}

int dpara_fuse_features(const dpara_config_t* cfg, const dpara_fusion_weights_t* fw, int32_t n_rows,
                        const void* hidden, void* feats, void* ws, size_t ws_bytes, void* stream) {
  int rc = check_cfg(cfg);
  if (rc) return rc;
  if (!fw) return fail(DPARA_E_INVALID, "fusion weights are NULL");
  CHECK_PTR(fw->fc, "fc");
  CHECK_PTR(fw->norm, "fusion norm");
  if (fw->n_feat < 1 || fw->n_feat > 8) return fail(DPARA_E_INVALID, "n_feat must be in [1, 8]");
  if (n_rows < 1) return fail(DPARA_E_INVALID, "n_rows must be >= 1");
  CHECK_PTR(hidden, "hidden");
  CHECK_PTR(feats, "feats");
  if (!aligned16(hidden) || !aligned16(feats)) return fail(DPARA_E_INVALID, "hidden and feats must be 16-byte aligned");
  if (!ws) return fail(DPARA_E_INVALID, "workspace is NULL");
  if (((uintptr_t)ws & 255u) != 0) return fail(DPARA_E_INVALID, "workspace must be 256-byte aligned");
  const size_t need = fuse_ws_bytes(cfg, n_rows);
  if (ws_bytes < need) return fail(DPARA_E_WORKSPACE, "workspace has %zu bytes, needs %zu", ws_bytes, need);
  if ((rc = check_device())) return rc;
  hipStream_t st = (hipStream_t)stream;
  const int H = cfg->hidden, K = fw->n_feat * cfg->hidden, dt = cfg->dtype;
  const int amode = dt == DPARA_BF16 ? A_BF16 : A_F32;
  const size_t esz = dt == DPARA_BF16 ? 2 : 4;
  float* planes = at<float>(ws, 256);
  for (int r0 = 0; r0 < n_rows; r0 += kFuseChunk) {
    const int m = n_rows - r0 < kFuseChunk ? n_rows - r0 : kFuseChunk;
    GemmArgs g{};
    g.A = (const char*)hidden + (size_t)r0 * K * esz;
    g.lda = K;
    g.B0 = g.B1 = g.B2 = fw->fc;
    g.n1 = g.n2 = H;
    g.M = m;
    g.N = H;
    g.K = K;
    g.C = planes;
    g.ldc = H;
    g.splits = gemm_splits(amode, EPI_STORE_F32, m, H, K);
    {
      Phase ph("fuse_gemm", st);
      HIP_TRY(launch_gemm(amode, EPI_STORE_F32, g, st), "fusion gemm");
    }
    // plane 0 stands in for the residual row; the other planes are added to it
    Phase ph("fuse_norm", st);
    HIP_TRY(launch_rmsnorm(dt, m, H, planes, m, 0, 0, planes + (size_t)m * H, g.splits - 1, (int64_t)m * H, 0,
                           fw->norm, cfg->rms_eps, (char*)feats + (size_t)r0 * H * esz, st),
            "fusion norm");
  }
  return DPARA_OK;
}

size_t dpara_branch_candidates_bytes(const dpara_config_t* cfg, int32_t batch) {
  if (check_cfg(cfg) || batch < 1) return 0;
  return head_cand_bytes(batch, cfg->gamma);
}

int dpara_branch_candidates(const dpara_config_t* cfg, const dpara_weights_t* w, int32_t batch, const float* reps,
                            void* cand, void* ws, size_t ws_bytes, void* stream) {
  int rc = check_cfg(cfg);
  if (rc) return rc;
  if (batch < 1) return fail(DPARA_E_INVALID, "batch must be >= 1");
  if (cfg->dtype != DPARA_BF16) return fail(DPARA_E_UNSUPPORTED, "branch candidates need a bf16 drafter");
  if (!head_prune_supported(1, cfg->gamma, cfg->vocab, cfg->ar_rank))
    return fail(DPARA_E_UNSUPPORTED, "branch candidates need ar_rank in {64, 128, 256}, vocab >= 64, gamma <= 63");
  if ((rc = check_weights(cfg, w, false))) return rc;
  CHECK_PTR(reps, "reps");
  CHECK_PTR(cand, "cand");
  if (!aligned16(reps)) return fail(DPARA_E_INVALID, "reps is not 16-byte aligned");
  if (((uintptr_t)cand & 255u) != 0) return fail(DPARA_E_INVALID, "cand must be 256-byte aligned");
  const Plan p = make_plan(cfg, batch, 64);
  if (!ws) return fail(DPARA_E_INVALID, "workspace is NULL");
  if (((uintptr_t)ws & 255u) != 0) return fail(DPARA_E_INVALID, "workspace must be 256-byte aligned");
  if (ws_bytes < p.total) return fail(DPARA_E_WORKSPACE, "workspace has %zu bytes, needs %zu", ws_bytes, p.total);
  if ((rc = check_device())) return rc;
  HIP_TRY(launch_branch_candidates(batch, cfg->gamma, cfg->hidden, cfg->vocab, cfg->ar_rank, reps, w->embed, w->ar_W,
                                   w->embed_norm2_max, cand, at<bf16_t>(ws, p.csplit), at<uint64_t>(ws, p.cpart),
                                   at<void>(ws, p.cscr), (hipStream_t)stream),
          "branch candidates");
  return DPARA_OK;
}

int dpara_candidates_prepare(const dpara_config_t* cfg, const dpara_weights_t* w, float* embed_norm2_max, void* ws,
                             size_t ws_bytes, void* stream) {
  int rc = check_cfg(cfg);
  if (rc) return rc;
  if (cfg->dtype != DPARA_BF16) return fail(DPARA_E_UNSUPPORTED, "branch candidates need a bf16 drafter");
  if (!w || !w->embed) return fail(DPARA_E_INVALID, "weights or embed is NULL");
  CHECK_PTR(embed_norm2_max, "embed_norm2_max");
  if (!ws || ((uintptr_t)ws & 255u) != 0) return fail(DPARA_E_INVALID, "workspace is NULL or not 256-byte aligned");
  const Plan p = make_plan(cfg, 1, 64);
  const size_t need = p.cscr + head_cand_scratch_bytes(1, cfg->gamma);
  if (ws_bytes < need) return fail(DPARA_E_WORKSPACE, "workspace has %zu bytes, needs %zu", ws_bytes, need);
  if ((rc = check_device())) return rc;
  HIP_TRY(launch_embed_prepare(w->embed, cfg->vocab, cfg->hidden, at<float>(ws, p.cscr), embed_norm2_max,
                               (hipStream_t)stream),
          "candidates prepare");
  return DPARA_OK;
}

int dpara_select_and_head_cand(const dpara_config_t* cfg, const dpara_weights_t* w, int32_t batch,
                               const float* reps, const void* cand, const int32_t* accept_len, const int32_t* bonus,
                               float* gathered, int32_t* drafts, int32_t* next_spine, float* margins, void* ws,
                               size_t ws_bytes, void* stream) {
  int rc = check_cfg(cfg);
  if (rc) return rc;
  if (batch < 1) return fail(DPARA_E_INVALID, "batch must be >= 1");
  if (cfg->dtype != DPARA_BF16) return fail(DPARA_E_UNSUPPORTED, "branch candidates need a bf16 drafter");
  if (!head_prune_supported(1, cfg->gamma, cfg->vocab, cfg->ar_rank))
    return fail(DPARA_E_UNSUPPORTED, "branch candidates need ar_rank in {64, 128, 256}, vocab >= 64, gamma <= 63");
  if ((rc = check_weights(cfg, w, false))) return rc;
  CHECK_PTR(reps, "reps");
  CHECK_PTR(cand, "cand");
  if (gathered && !aligned16(gathered)) return fail(DPARA_E_INVALID, "gathered is not 16-byte aligned");
  if (!accept_len || !bonus || !drafts || !next_spine)
    return fail(DPARA_E_INVALID, "accept_len, bonus, drafts and next_spine must be non-NULL");
  const Plan p = make_plan(cfg, batch, 64);
  if (!ws) return fail(DPARA_E_INVALID, "workspace is NULL");
  if (((uintptr_t)ws & 255u) != 0) return fail(DPARA_E_INVALID, "workspace must be 256-byte aligned");
  const size_t need = p.hwpart + up256((size_t)head_prune_wparts() * 4);
  if (ws_bytes < need) return fail(DPARA_E_WORKSPACE, "workspace has %zu bytes, needs %zu", ws_bytes, need);
  if ((rc = check_device())) return rc;

  hipStream_t st = (hipStream_t)stream;
  const int g = cfg->gamma, H = cfg->hidden, V = cfg->vocab;
  int* status = at<int>(ws, 0);
  int* hflag = at<int>(ws, p.hflag);
  bf16_t* Gs = at<bf16_t>(ws, p.Gsplit);
  HIP_TRY(launch_gather_branch(batch, g, H, reps, accept_len, at<float>(ws, p.G), gathered, Gs,
                               at<uint64_t>(ws, p.arpart), (int64_t)2 * 16 * p.ar_grid * 2, status, st),
          "gather_branch");
  HIP_TRY(launch_head_from_candidates(batch, g, V, cfg->ar_rank, cand, w->ar_E, w->ar_W, accept_len, bonus, drafts,
                                      next_spine, margins, hflag, status, st),
          "pruned head");
  // Only if some step was not proven: the LM head over the gathered rows and the full head
  // (both return at once otherwise).
  GemmArgs lm{};
  lm.A = Gs;
  lm.lo_off = (int64_t)batch * g * H;
  lm.lda = H;
  lm.B0 = lm.B1 = lm.B2 = w->embed;
  lm.n1 = lm.n2 = V;
  lm.M = batch * g;
  lm.N = V;
  lm.K = H;
  lm.C = at<void>(ws, p.logits);
  lm.ldc = V;
  lm.only_if = hflag;
  {
    Phase ph("lm_head", st);
    HIP_TRY(launch_gemm(A_BF16_DUAL, EPI_STORE_F32, lm, st), "lm head gemm");
  }
  HIP_TRY(launch_ar_head(cfg->dtype, batch, g, V, cfg->ar_rank, at<float>(ws, p.logits), w->ar_E, w->ar_W, bonus,
                         drafts, next_spine, margins, at<uint64_t>(ws, p.hpart), p.h_chunks, p.h_chunk,
                         p.ar_grid ? at<uint64_t>(ws, p.arpart) : nullptr, p.ar_grid, status, hflag, st),
          "ar head");
  return DPARA_OK;
}

}  // extern "C"
