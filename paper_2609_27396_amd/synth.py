"""Seeded synthetic inputs for the DPara drafter hot path.

This module only draws random numbers and lays them out; it holds none of the
method's arithmetic.  Both the GPU path (through tests and the benchmark) and
the CPU oracle consume what it produces, so it is the single shared source of
inputs.

Stream contract: every tensor is split into chunks of ``CHUNK`` elements and
chunk ``c`` of the tensor with stable id ``tid`` is filled from
``PCG64(SeedSequence(seed, spawn_key=(tid, c)))`` with ``standard_normal``
in float32, then scaled.  The values therefore do not depend on generation
order or thread count.  In bf16 mode matrices and embeddings are rounded to
bfloat16 (round-to-nearest-even) on the host so that both sides see
bit-identical weights.

Shapes follow the paper's setting (Section 4.1: Qwen3-8B and Qwen3-14B
targets, drafts of length d scored per round, batch 1..16); the acceptance
regime (accepted length ~ Geometric, capped at the draft length) and the
planted target logits are a reading of this module: the paper reports mean
accepted lengths but not their distribution.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field, replace

import numpy as np

CHUNK = 1 << 22


# ----------------------------------------------------------------------------
# shapes and workloads
# ----------------------------------------------------------------------------
@dataclass(frozen=True)
class DrafterShape:
    n_layers: int
    hidden: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    ffn: int
    vocab: int
    gamma: int          # draft length (d in the paper's Algorithm 1)
    ar_rank: int        # rank of the AR head's token embedding E
    qk_norm: bool
    dtype: str          # "f32" or "bf16"
    rms_eps: float = 1e-6
    rope_base: float = 1e6

    @property
    def rows(self) -> int:
        """Query rows per request: (gamma+1) spine rows + (gamma+1)*gamma mask rows."""
        return (self.gamma + 1) ** 2


@dataclass(frozen=True)
class Workload:
    name: str
    shape: DrafterShape
    batch: int
    ctx_min: int            # context lengths drawn uniformly in [ctx_min, ctx_max]
    ctx_max: int
    p_reject: float         # per-draft rejection probability (accepted length ~ Geometric)
    seed_w: int = 0
    seed_in: int = 1
    logits_dtype: str = "bf16"
    description: str = ""


TINY = DrafterShape(n_layers=1, hidden=256, n_q_heads=4, n_kv_heads=2, head_dim=64, ffn=704,
                    vocab=1024, gamma=4, ar_rank=256, qk_norm=False, dtype="f32")
QWEN3_8B = DrafterShape(n_layers=5, hidden=4096, n_q_heads=32, n_kv_heads=8, head_dim=128,
                        ffn=12288, vocab=151936, gamma=16, ar_rank=256, qk_norm=True, dtype="bf16")
# The 36-layer Qwen3-8B-shaped target used for the single-GPU full round (timing only).
QWEN3_8B_TARGET = DrafterShape(n_layers=36, hidden=4096, n_q_heads=32, n_kv_heads=8, head_dim=128,
                               ffn=12288, vocab=151936, gamma=16, ar_rank=256, qk_norm=True, dtype="bf16")
QWEN3_14B = DrafterShape(n_layers=5, hidden=5120, n_q_heads=40, n_kv_heads=8, head_dim=128,
                         ffn=17408, vocab=151936, gamma=16, ar_rank=256, qk_norm=True, dtype="bf16")

WORKLOADS = {
    "tiny": Workload("tiny", TINY, batch=1, ctx_min=128, ctx_max=128, p_reject=0.3,
                     seed_w=0, seed_in=0, logits_dtype="f32",
                     description="1-layer 256-wide fp32 drafter, gamma=4, context 128, batch 1"),
    "qwen3_8b_b1": Workload("qwen3_8b_b1", QWEN3_8B, batch=1, ctx_min=2048, ctx_max=2048,
                            p_reject=0.2,
                            description="Qwen3-8B-shaped 5-layer bf16 drafter, gamma=16, "
                                        "context 2048, batch 1"),
    "qwen3_8b_b16": Workload("qwen3_8b_b16", QWEN3_8B, batch=16, ctx_min=512, ctx_max=4096,
                             p_reject=0.2,
                             description="Qwen3-8B-shaped drafter, gamma=16, batch 16, ragged "
                                         "contexts U[512,4096]"),
    "full_round": Workload("full_round", QWEN3_8B, batch=16, ctx_min=2048, ctx_max=2048, p_reject=0.2,
                           description="full round on one GPU: 36-layer Qwen3-8B-shaped random target "
                                       "verifying gamma=16 blocks at batch 16, contexts 2048, with the "
                                       "5-layer drafter's backbone on a concurrent stream"),
    "qwen3_14b_b8": Workload("qwen3_14b_b8", QWEN3_14B, batch=8, ctx_min=8192, ctx_max=8192,
                             p_reject=0.2,
                             description="Qwen3-14B-shaped 5-layer bf16 drafter, gamma=16, "
                                         "context 8192, batch 8"),
}


# ----------------------------------------------------------------------------
# bf16 helpers (input preparation only)
# ----------------------------------------------------------------------------
def to_bf16_values(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even); float32 out."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    u = (u + (np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1)))) & np.uint32(0xFFFF0000)
    return u.view(np.float32)


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """Upper 16 bits of float32 values that are already bfloat16-representable."""
    return (np.ascontiguousarray(x, dtype=np.float32).view(np.uint32) >> np.uint32(16)).astype(np.uint16)


# ----------------------------------------------------------------------------
# chunked, order-independent normal streams
# ----------------------------------------------------------------------------
def _threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def _fill_chunk(out: np.ndarray, seed: int, tid: int, c: int, std: float):
    g = np.random.Generator(np.random.PCG64(np.random.SeedSequence(seed, spawn_key=(tid, c))))
    g.standard_normal(out=out, dtype=np.float32)
    if std != 1.0:
        out *= np.float32(std)


def normal_tensors(specs, seed: int) -> list:
    """specs: list of (tid, shape, std, mean, round_bf16).  Returns float32 arrays."""
    outs, jobs = [], []
    for tid, shape, std, mean, rb in specs:
        a = np.empty(shape, np.float32)
        flat = a.reshape(-1)
        for c in range(0, max(1, (flat.size + CHUNK - 1) // CHUNK)):
            jobs.append((flat[c * CHUNK:(c + 1) * CHUNK], tid, c, std))
        outs.append((a, mean, rb))
    with ThreadPoolExecutor(_threads()) as ex:
        list(ex.map(lambda j: _fill_chunk(j[0], seed, j[1], j[2], j[3]), jobs))
    res = []
    for a, mean, rb in outs:
        if mean != 0.0:
            a += np.float32(mean)
        if rb:
            flat = a.reshape(-1)
            for s in range(0, flat.size, CHUNK):
                flat[s:s + CHUNK] = to_bf16_values(flat[s:s + CHUNK])
        res.append(a)
    return res


# ----------------------------------------------------------------------------
# weights
# ----------------------------------------------------------------------------
LAYER_KEYS = ("attn_norm", "wq", "wk", "wv", "q_norm", "k_norm", "wo", "mlp_norm",
              "w_gate", "w_up", "w_down")


def weight_specs(s: DrafterShape, gain_jitter: float = 0.0, weight_std: float = 0.02,
                 ar_e_std: float = 0.02, ar_w_std: float = 0.02):
    """(name, tid, shape, std, mean, round_bf16) for every drafter parameter."""
    bf = s.dtype == "bf16"
    H, hd, F, V = s.hidden, s.head_dim, s.ffn, s.vocab
    gain = (gain_jitter, 1.0, False)  # norm gains stay float32 in every mode
    out = [("embed", 1, (V, H), weight_std, 0.0, bf),
           ("mask_emb", 2, (H,), weight_std, 0.0, bf),
           ("final_norm", 3, (H,)) + gain,
           ("ar_E", 4, (V, s.ar_rank), ar_e_std, 0.0, bf),
           ("ar_W", 5, (V, s.ar_rank), ar_w_std, 0.0, bf)]
    for l in range(s.n_layers):
        b = 100 + 16 * l
        out += [(f"L{l}.attn_norm", b + 0, (H,)) + gain,
                (f"L{l}.wq", b + 1, (s.n_q_heads * hd, H), weight_std, 0.0, bf),
                (f"L{l}.wk", b + 2, (s.n_kv_heads * hd, H), weight_std, 0.0, bf),
                (f"L{l}.wv", b + 3, (s.n_kv_heads * hd, H), weight_std, 0.0, bf),
                (f"L{l}.q_norm", b + 4, (hd,)) + gain,
                (f"L{l}.k_norm", b + 5, (hd,)) + gain,
                (f"L{l}.wo", b + 6, (H, s.n_q_heads * hd), weight_std, 0.0, bf),
                (f"L{l}.mlp_norm", b + 7, (H,)) + gain,
                (f"L{l}.w_gate", b + 8, (F, H), weight_std, 0.0, bf),
                (f"L{l}.w_up", b + 9, (F, H), weight_std, 0.0, bf),
                (f"L{l}.w_down", b + 10, (H, F), weight_std, 0.0, bf)]
    return out


def make_weights(s: DrafterShape, seed: int = 0, **kw) -> dict:
    """All drafter parameters as float32 numpy arrays (bf16-valued in bf16 mode).

    Norm gains are exactly 1 unless ``gain_jitter`` > 0 (tests use jitter so that
    a gain applied in the wrong place shows up)."""
    specs = weight_specs(s, **kw)
    arrs = normal_tensors([(tid, shp, std, mean, rb) for _, tid, shp, std, mean, rb in specs], seed)
    return {name: a for (name, *_), a in zip(specs, arrs)}


def make_target_weights(s: DrafterShape, seed: int = 100, **kw) -> dict:
    """A random target of the same layer structure: drafter-style layer weights, token
    embedding, final norm and an untied LM head `lm_head` [V, H] (N(0, weight_std))."""
    w = make_weights(s, seed=seed, **kw)
    for k in ("mask_emb", "ar_E", "ar_W"):
        w.pop(k)
    std = kw.get("weight_std", 0.02)
    (lm,) = normal_tensors([(6, (s.vocab, s.hidden), std, 0.0, s.dtype == "bf16")], seed)
    w["lm_head"] = lm
    return w


def make_fusion_weights(s: DrafterShape, n_feat: int = 3, seed: int = 0, gain_jitter: float = 0.0,
                        weight_std: float = 0.02) -> dict:
    """The feature-fusion projection `fc` [H, n_feat*H] (N(0, weight_std), bf16-valued in
    bf16 mode) and its RMSNorm gain `fc_norm` [H] (float32)."""
    fc, g = normal_tensors([(7, (s.hidden, n_feat * s.hidden), weight_std, 0.0, s.dtype == "bf16"),
                            (8, (s.hidden,), gain_jitter, 1.0, False)], seed)
    return {"fc": fc, "fc_norm": g}


def make_target_hidden(s: DrafterShape, n_rows: int, n_feat: int = 3, seed: int = 1,
                       std: float = 1.0) -> np.ndarray:
    """Concatenated target hidden states [n_rows, n_feat*H] of the rows to be fused,
    N(0, std) (bf16-valued in bf16 mode)."""
    (h,) = normal_tensors([(9, (n_rows, n_feat * s.hidden), std, 0.0, s.dtype == "bf16")], seed)
    return h


def make_target_cache(s: DrafterShape, ctx_lens, seed: int = 101):
    """The target's own per-layer context K/V: k[l][b], v[l][b] of shape [n_b, n_kv, hd],
    N(0, 1) (bf16-valued in bf16 mode)."""
    bf = s.dtype == "bf16"
    specs, keys = [], []
    for l in range(s.n_layers):
        for b, n in enumerate(ctx_lens):
            for kind in (0, 1):
                specs.append((5000 + 64 * l + 2 * b + kind, (int(n), s.n_kv_heads, s.head_dim), 1.0, 0.0, bf))
                keys.append((l, b, kind))
    arrs = normal_tensors(specs, seed)
    k = [[None] * len(ctx_lens) for _ in range(s.n_layers)]
    v = [[None] * len(ctx_lens) for _ in range(s.n_layers)]
    for (l, b, kind), a in zip(keys, arrs):
        (k if kind == 0 else v)[l][b] = a
    return k, v


def device_normal_(t, seed: int, std: float = 1.0):
    """Fill a device tensor in place with seeded N(0, std) draws (device generator; used for
    the large timing-only target, which has no oracle)."""
    import torch
    g = torch.Generator(device=t.device)
    g.manual_seed(int(seed))
    tmp = torch.empty(t.shape, dtype=torch.float32, device=t.device)
    tmp.normal_(0.0, std, generator=g)
    t.copy_(tmp)
    return t


# ----------------------------------------------------------------------------
# per-round inputs
# ----------------------------------------------------------------------------
@dataclass
class RoundInputs:
    ctx_lens: np.ndarray             # [B] int32
    ctx_feats: list                  # B arrays [n_b, H] float32 (fused target features)
    spine: np.ndarray                # [B, gamma+1] int32: t_0 = previous bonus, t_1..t_gamma drafts
    accept_planted: np.ndarray       # [B] int32: accepted length the planted logits encode
    bonus_planted: np.ndarray        # [B] int32
    target_logits: np.ndarray        # [B, gamma+1, V] float32 (bf16-valued if logits_dtype bf16)
    new_feats: np.ndarray            # [B, gamma+1, H] float32: features of t_{0:gamma} (append input)
    extra: dict = field(default_factory=dict)


def _rng(seed: int, key: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(seed, spawn_key=(key,))))


def accepted_lengths(rng: np.random.Generator, batch: int, gamma: int, p: float) -> np.ndarray:
    """r = min(G-1, gamma) with G ~ Geometric(p) on {1,2,...}."""
    return np.minimum(rng.geometric(p, size=batch) - 1, gamma).astype(np.int32)


def plant_target_logits(rng: np.random.Generator, spine: np.ndarray, accept: np.ndarray,
                        vocab: int, bf16: bool):
    """Target logits whose greedy verdict is exactly (accept, bonus).

    Rows are N(0,1).  For j < r the draft t_{j+1} is made the unique row maximum;
    at j = r a bonus different from t_{r+1} (any token when r = gamma) is made the
    unique maximum.  Rows after r are left random.  Returns (logits, bonus)."""
    B, G1 = spine.shape
    gamma = G1 - 1
    T = rng.standard_normal((B, G1, vocab), dtype=np.float32)
    if bf16:
        T = to_bf16_values(T)
    bonus = np.zeros(B, np.int32)
    for b in range(B):
        r = int(accept[b])
        for j in range(r + 1):
            if j < r:
                tok = int(spine[b, j + 1])
            else:
                tok = int(rng.integers(0, vocab))
                if r < gamma:
                    while tok == int(spine[b, r + 1]):
                        tok = int(rng.integers(0, vocab))
                bonus[b] = tok
            top = np.float32(T[b, j].max()) + np.float32(1.0)
            if bf16:
                top = to_bf16_values(np.array([top], np.float32))[0]
            T[b, j, tok] = top
    return T, bonus


def make_round(w: Workload, seed: int | None = None, ctx_lens=None) -> RoundInputs:
    s = w.shape
    seed = w.seed_in if seed is None else seed
    rng = _rng(seed, 1000)
    B, H, G1 = w.batch, s.hidden, s.gamma + 1
    if ctx_lens is None:
        ctx_lens = rng.integers(w.ctx_min, w.ctx_max + 1, size=B).astype(np.int32)
    ctx_lens = np.asarray(ctx_lens, np.int32)
    bf = s.dtype == "bf16"
    specs = [(2000 + b, (int(ctx_lens[b]), H), 1.0, 0.0, bf) for b in range(B)]
    specs.append((3000, (B, G1, H), 1.0, 0.0, bf))
    arrs = normal_tensors(specs, seed)
    spine = rng.integers(0, s.vocab, size=(B, G1)).astype(np.int32)
    accept = accepted_lengths(rng, B, s.gamma, w.p_reject)
    T, bonus = plant_target_logits(rng, spine, accept, s.vocab, w.logits_dtype == "bf16")
    return RoundInputs(ctx_lens=ctx_lens, ctx_feats=arrs[:B], spine=spine, accept_planted=accept,
                       bonus_planted=bonus, target_logits=T, new_feats=arrs[B])


def shrink(shape: DrafterShape, **kw) -> DrafterShape:
    return replace(shape, **kw)
