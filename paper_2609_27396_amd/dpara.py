"""Python binding of libdpara (include/dpara.h): argument marshalling only.

The functions named like the C entry points take the same arguments (device
pointers as ints, ctypes structs, the stream handle) and raise ``DparaError``
on a non-zero return.  ``DeviceDrafter`` / ``DeviceContext`` own the device
tensors (allocated with PyTorch) that back the C structs.  Every step of the
path runs in the HIP kernels of libdpara.so; when the library is missing,
``lib()`` raises instead of falling back to anything else.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# DPARA_LIB_PATH selects another build of the same library (the tests load the host-sanitized
# libdpara_asan.so through it); the default is the in-tree libdpara.so.
LIB_PATH = os.environ.get("DPARA_LIB_PATH") or os.path.join(_HERE, "libdpara.so")

DPARA_OK, DPARA_E_INVALID, DPARA_E_UNSUPPORTED, DPARA_E_WORKSPACE, DPARA_E_CAPACITY, DPARA_E_HIP = 0, -1, -2, -3, -4, -5
DPARA_F32, DPARA_BF16 = 0, 1
STATUS_TOKEN_RANGE, STATUS_CTX_FULL, STATUS_VERDICT_RANGE, STATUS_COUNT_RANGE, STATUS_HEAD_TIMEOUT = 1, 2, 4, 8, 16

EXPORTS = ("dpara_workspace_bytes", "dpara_ctx_append", "dpara_backbone_all_boundaries",
           "dpara_verify_greedy", "dpara_select_and_head", "dpara_branch_candidates_bytes",
           "dpara_branch_candidates", "dpara_select_and_head_cand", "dpara_clear_status",
           "dpara_last_error", "dpara_version", "dpara_profile_enable", "dpara_profile_read",
           "dpara_target_workspace_bytes", "dpara_target_forward", "dpara_target_forward_hidden",
           "dpara_fuse_workspace_bytes", "dpara_fuse_features", "dpara_select_and_head_sampled",
           "dpara_verify_sampled", "dpara_head_prepare", "dpara_backbone_trace",
           "dpara_verify_greedy_noalloc", "dpara_candidates_prepare")

PHASES = ("append_gemm", "append_store", "assemble", "rmsnorm", "qkv_gemm", "qk_norm_rope", "attn_ctx",
          "attn_merge", "o_gemm", "gateup_gemm", "down_gemm", "final_norm", "verify", "gather", "lm_head",
          "ar_step", "fuse_gemm", "fuse_norm")


class DparaError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"dpara error {code}: {msg}")
        self.code = code


class DparaConfig(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("hidden", ctypes.c_int32), ("n_q_heads", ctypes.c_int32),
                ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32), ("ffn", ctypes.c_int32),
                ("vocab", ctypes.c_int32), ("gamma", ctypes.c_int32), ("ar_rank", ctypes.c_int32),
                ("qk_norm", ctypes.c_int32), ("dtype", ctypes.c_int32), ("rms_eps", ctypes.c_float),
                ("rope_base", ctypes.c_float)]


class DparaLayerWeights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in ("attn_norm", "wq", "wk", "wv", "q_norm", "k_norm", "wo",
                                               "mlp_norm", "w_gate", "w_up", "w_down")]


class DparaWeights(ctypes.Structure):
    _fields_ = [("embed", ctypes.c_void_p), ("mask_emb", ctypes.c_void_p), ("final_norm", ctypes.c_void_p),
                ("ar_E", ctypes.c_void_p), ("ar_W", ctypes.c_void_p),
                ("layers", ctypes.POINTER(DparaLayerWeights)), ("ar_w_norm2_max", ctypes.c_void_p),
                ("embed_norm2_max", ctypes.c_void_p)]


class DparaTargetWeights(ctypes.Structure):
    _fields_ = [("embed", ctypes.c_void_p), ("lm_head", ctypes.c_void_p), ("final_norm", ctypes.c_void_p),
                ("layers", ctypes.POINTER(DparaLayerWeights))]


class DparaFusionWeights(ctypes.Structure):
    _fields_ = [("fc", ctypes.c_void_p), ("norm", ctypes.c_void_p), ("n_feat", ctypes.c_int32)]


class DparaCtx(ctypes.Structure):
    _fields_ = [("k", ctypes.c_void_p), ("v", ctypes.c_void_p), ("ctx_len", ctypes.c_void_p),
                ("batch_cap", ctypes.c_int32), ("ctx_cap", ctypes.c_int32)]


_lib = None


def lib():
    """Load libdpara.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2609_27396_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        P, I32, SZ, VP = ctypes.POINTER, ctypes.c_int32, ctypes.c_size_t, ctypes.c_void_p
        L.dpara_workspace_bytes.argtypes = [P(DparaConfig), I32, I32]
        L.dpara_workspace_bytes.restype = SZ
        L.dpara_ctx_append.argtypes = [P(DparaConfig), P(DparaWeights), P(DparaCtx), I32, VP, VP, I32, VP, SZ, VP]
        L.dpara_backbone_all_boundaries.argtypes = [P(DparaConfig), P(DparaWeights), P(DparaCtx), I32, VP, VP, VP,
                                                    SZ, VP]
        L.dpara_backbone_trace.argtypes = [P(DparaConfig), P(DparaWeights), P(DparaCtx), I32, VP, VP, VP, VP, SZ,
                                           VP]
        L.dpara_verify_greedy.argtypes = [P(DparaConfig), I32, VP, I32, VP, VP, VP, VP, VP, SZ, VP]
        L.dpara_verify_greedy_noalloc.argtypes = [P(DparaConfig), I32, VP, I32, VP, VP, VP, VP, VP, VP]
        L.dpara_select_and_head.argtypes = [P(DparaConfig), P(DparaWeights), I32, VP, VP, VP, VP, VP, VP, VP, VP,
                                            SZ, VP]
        L.dpara_branch_candidates_bytes.argtypes = [P(DparaConfig), I32]
        L.dpara_branch_candidates_bytes.restype = SZ
        L.dpara_branch_candidates.argtypes = [P(DparaConfig), P(DparaWeights), I32, VP, VP, VP, SZ, VP]
        L.dpara_select_and_head_cand.argtypes = [P(DparaConfig), P(DparaWeights), I32, VP, VP, VP, VP, VP, VP, VP,
                                                 VP, VP, SZ, VP]
        L.dpara_clear_status.argtypes = [VP, VP]
        L.dpara_target_workspace_bytes.argtypes = [P(DparaConfig), I32, I32]
        L.dpara_target_workspace_bytes.restype = SZ
        L.dpara_target_forward.argtypes = [P(DparaConfig), P(DparaTargetWeights), P(DparaCtx), I32, VP, VP, I32,
                                           VP, SZ, VP]
        L.dpara_target_forward_hidden.argtypes = [P(DparaConfig), P(DparaTargetWeights), P(DparaCtx), I32, VP, VP,
                                                  I32, P(I32), I32, VP, VP, SZ, VP]
        L.dpara_fuse_workspace_bytes.argtypes = [P(DparaConfig), I32, I32]
        L.dpara_fuse_workspace_bytes.restype = SZ
        L.dpara_fuse_features.argtypes = [P(DparaConfig), P(DparaFusionWeights), I32, VP, VP, VP, SZ, VP]
        F32, U64 = ctypes.c_float, ctypes.c_uint64
        L.dpara_select_and_head_sampled.argtypes = [P(DparaConfig), P(DparaWeights), I32, VP, VP, VP, VP, VP, VP,
                                                    VP, F32, U64, VP, VP, VP, SZ, VP]
        L.dpara_verify_sampled.argtypes = [P(DparaConfig), I32, VP, I32, VP, VP, F32, U64, VP, VP, VP, VP, SZ, VP]
        L.dpara_head_prepare.argtypes = [P(DparaConfig), P(DparaWeights), VP, VP, SZ, VP]
        L.dpara_candidates_prepare.argtypes = [P(DparaConfig), P(DparaWeights), VP, VP, SZ, VP]
        L.dpara_last_error.restype = ctypes.c_char_p
        L.dpara_version.restype = I32
        L.dpara_profile_enable.argtypes = [I32]
        L.dpara_profile_read.argtypes = [ctypes.c_char_p, P(ctypes.c_double), P(ctypes.c_int64)]
        for name in ("dpara_ctx_append", "dpara_backbone_all_boundaries", "dpara_verify_greedy",
                     "dpara_select_and_head", "dpara_branch_candidates", "dpara_select_and_head_cand",
                     "dpara_clear_status", "dpara_profile_enable",
                     "dpara_profile_read", "dpara_target_forward", "dpara_fuse_features",
                     "dpara_target_forward_hidden", "dpara_select_and_head_sampled", "dpara_verify_sampled",
                     "dpara_head_prepare", "dpara_backbone_trace", "dpara_verify_greedy_noalloc",
                     "dpara_candidates_prepare"):
            getattr(L, name).restype = ctypes.c_int
        _lib = L
    return _lib


def _check(rc: int):
    if rc != DPARA_OK:
        raise DparaError(rc, lib().dpara_last_error().decode())


def _ref(x):
    return ctypes.byref(x) if x is not None else None


# ---------------------------------------------------------------- raw entry points
def dpara_workspace_bytes(cfg: DparaConfig, batch: int, ctx_cap: int) -> int:
    return int(lib().dpara_workspace_bytes(ctypes.byref(cfg), batch, ctx_cap))


def dpara_ctx_append(cfg, w, ctx, batch, feats, n_new, n_max, ws, ws_bytes, stream):
    _check(lib().dpara_ctx_append(_ref(cfg), _ref(w), _ref(ctx), batch, feats, n_new, n_max, ws, ws_bytes, stream))


def dpara_backbone_all_boundaries(cfg, w, ctx, batch, spine, reps, ws, ws_bytes, stream):
    _check(lib().dpara_backbone_all_boundaries(_ref(cfg), _ref(w), _ref(ctx), batch, spine, reps, ws, ws_bytes,
                                               stream))


def dpara_verify_greedy(cfg, batch, target_logits, logits_dtype, spine, accept_len, bonus, target_argmax, ws,
                        ws_bytes, stream):
    _check(lib().dpara_verify_greedy(_ref(cfg), batch, target_logits, logits_dtype, spine, accept_len, bonus,
                                     target_argmax, ws, ws_bytes, stream))


def dpara_select_and_head(cfg, w, batch, reps, accept_len, bonus, gathered, drafts, next_spine, margins, ws,
                          ws_bytes, stream):
    _check(lib().dpara_select_and_head(_ref(cfg), _ref(w), batch, reps, accept_len, bonus, gathered, drafts,
                                       next_spine, margins, ws, ws_bytes, stream))


def dpara_branch_candidates_bytes(cfg: DparaConfig, batch: int) -> int:
    return int(lib().dpara_branch_candidates_bytes(_ref(cfg), batch))


def dpara_branch_candidates(cfg, w, batch, reps, cand, ws, ws_bytes, stream):
    _check(lib().dpara_branch_candidates(_ref(cfg), _ref(w), batch, reps, cand, ws, ws_bytes, stream))


def dpara_select_and_head_cand(cfg, w, batch, reps, cand, accept_len, bonus, gathered, drafts, next_spine, margins,
                               ws, ws_bytes, stream):
    _check(lib().dpara_select_and_head_cand(_ref(cfg), _ref(w), batch, reps, cand, accept_len, bonus, gathered,
                                            drafts, next_spine, margins, ws, ws_bytes, stream))


def dpara_target_workspace_bytes(cfg: DparaConfig, batch: int, ctx_cap: int) -> int:
    return int(lib().dpara_target_workspace_bytes(ctypes.byref(cfg), batch, ctx_cap))


def dpara_target_forward(cfg, w, ctx, batch, block, logits, logits_dtype, ws, ws_bytes, stream):
    _check(lib().dpara_target_forward(_ref(cfg), _ref(w), _ref(ctx), batch, block, logits, logits_dtype, ws,
                                      ws_bytes, stream))


def dpara_clear_status(ws, stream):
    _check(lib().dpara_clear_status(ws, stream))


def dpara_last_error() -> str:
    return lib().dpara_last_error().decode()


def dpara_version() -> int:
    return int(lib().dpara_version())


def dpara_profile_enable(on: bool):
    _check(lib().dpara_profile_enable(int(bool(on))))


def dpara_profile_read(phase: str):
    """(total_ms, launches) recorded for `phase` since the last enable."""
    t, n = ctypes.c_double(), ctypes.c_int64()
    _check(lib().dpara_profile_read(phase.encode(), ctypes.byref(t), ctypes.byref(n)))
    return t.value, n.value


# ---------------------------------------------------------------- config helpers
def make_config(shape) -> DparaConfig:
    """DparaConfig from an object with the DrafterShape fields."""
    return DparaConfig(n_layers=shape.n_layers, hidden=shape.hidden, n_q_heads=shape.n_q_heads,
                       n_kv_heads=shape.n_kv_heads, head_dim=shape.head_dim, ffn=shape.ffn, vocab=shape.vocab,
                       gamma=shape.gamma, ar_rank=shape.ar_rank, qk_norm=int(bool(shape.qk_norm)),
                       dtype=DPARA_BF16 if shape.dtype == "bf16" else DPARA_F32, rms_eps=shape.rms_eps,
                       rope_base=shape.rope_base)


def _ptr(t) -> int:
    return 0 if t is None else int(t.data_ptr())


def _stream(stream) -> int:
    import torch
    if stream is None:
        return int(torch.cuda.current_stream().cuda_stream)
    return int(getattr(stream, "cuda_stream", stream))


# ---------------------------------------------------------------- device holders
class DeviceDrafter:
    """Drafter weights resident in HBM plus the C structs that point at them."""

    def __init__(self, shape, weights: dict, device="cuda"):
        import torch
        self.shape = shape
        self.cfg = make_config(shape)
        self.device = device
        mat_dtype = torch.bfloat16 if shape.dtype == "bf16" else torch.float32
        self.t = {}
        for name, arr in weights.items():
            base = name.split(".")[-1]
            is_gain = base in ("attn_norm", "mlp_norm", "q_norm", "k_norm", "final_norm")
            src = torch.from_numpy(np.ascontiguousarray(arr))
            self.t[name] = src.to(device=device, dtype=torch.float32 if is_gain else mat_dtype)
        L = shape.n_layers
        self._layers = (DparaLayerWeights * L)()
        for l in range(L):
            for f in ("attn_norm", "wq", "wk", "wv", "q_norm", "k_norm", "wo", "mlp_norm", "w_gate", "w_up",
                      "w_down"):
                setattr(self._layers[l], f, _ptr(self.t[f"L{l}.{f}"]))
        self.w = DparaWeights(embed=_ptr(self.t["embed"]), mask_emb=_ptr(self.t["mask_emb"]),
                              final_norm=_ptr(self.t["final_norm"]), ar_E=_ptr(self.t["ar_E"]),
                              ar_W=_ptr(self.t["ar_W"]),
                              layers=ctypes.cast(self._layers, ctypes.POINTER(DparaLayerWeights)))

    @property
    def mat_dtype(self):
        import torch
        return torch.bfloat16 if self.shape.dtype == "bf16" else torch.float32

    def prepare_head(self, ws, stream=None):
        """Compute max_v |ar_W[v]|^2 once (dpara_head_prepare) and point the weights at it, so
        head calls skip their own pass over ar_W."""
        import torch
        self.norm2 = torch.empty(1, dtype=torch.float32, device=self.device)
        _check(lib().dpara_head_prepare(_ref(self.cfg), _ref(self.w), _ptr(self.norm2), ws.ptr, ws.nbytes,
                                        _stream(stream)))
        self.w.ar_w_norm2_max = _ptr(self.norm2)

    def unprepare_head(self):
        self.w.ar_w_norm2_max = None

    def prepare_candidates(self, ws, stream=None):
        """Compute max_v |embed[v]|^2 once (dpara_candidates_prepare) and point the weights at
        it, so dpara_branch_candidates calls skip their own pass over the embedding."""
        import torch
        self.enorm2 = torch.empty(1, dtype=torch.float32, device=self.device)
        _check(lib().dpara_candidates_prepare(_ref(self.cfg), _ref(self.w), _ptr(self.enorm2), ws.ptr, ws.nbytes,
                                              _stream(stream)))
        self.w.embed_norm2_max = _ptr(self.enorm2)

    def unprepare_candidates(self):
        self.w.embed_norm2_max = None


class DeviceTarget:
    """Target weights resident in HBM (from host arrays, or generated on device when
    `weights` is None: timing-only)."""

    def __init__(self, shape, weights: dict | None, device="cuda", seed: int = 100):
        import torch
        from . import synth
        self.shape = shape
        self.cfg = make_config(shape)
        self.cfg.ar_rank = 64
        bf = torch.bfloat16
        H, hd, F, V = shape.hidden, shape.head_dim, shape.ffn, shape.vocab
        nq, nkv = shape.n_q_heads, shape.n_kv_heads
        self.t = {}
        if weights is not None:
            for name, arr in weights.items():
                base = name.split(".")[-1]
                is_gain = base in ("attn_norm", "mlp_norm", "q_norm", "k_norm", "final_norm")
                self.t[name] = torch.from_numpy(np.ascontiguousarray(arr)).to(
                    device=device, dtype=torch.float32 if is_gain else bf)
        else:
            shapes = {"embed": (V, H), "lm_head": (V, H)}
            for l in range(shape.n_layers):
                shapes.update({f"L{l}.wq": (nq * hd, H), f"L{l}.wk": (nkv * hd, H), f"L{l}.wv": (nkv * hd, H),
                               f"L{l}.wo": (H, nq * hd), f"L{l}.w_gate": (F, H), f"L{l}.w_up": (F, H),
                               f"L{l}.w_down": (H, F)})
            for i, (name, shp) in enumerate(sorted(shapes.items())):
                self.t[name] = synth.device_normal_(torch.empty(shp, dtype=bf, device=device), seed * 1000 + i, 0.02)
            ones = lambda n: torch.ones(n, dtype=torch.float32, device=device)
            self.t["final_norm"] = ones(H)
            for l in range(shape.n_layers):
                for g, n in (("attn_norm", H), ("mlp_norm", H), ("q_norm", hd), ("k_norm", hd)):
                    self.t[f"L{l}.{g}"] = ones(n)
        self._layers = (DparaLayerWeights * shape.n_layers)()
        for l in range(shape.n_layers):
            for f in ("attn_norm", "wq", "wk", "wv", "q_norm", "k_norm", "wo", "mlp_norm", "w_gate", "w_up",
                      "w_down"):
                setattr(self._layers[l], f, _ptr(self.t[f"L{l}.{f}"]))
        self.w = DparaTargetWeights(embed=_ptr(self.t["embed"]), lm_head=_ptr(self.t["lm_head"]),
                                    final_norm=_ptr(self.t["final_norm"]),
                                    layers=ctypes.cast(self._layers, ctypes.POINTER(DparaLayerWeights)))


class DeviceContext:
    """Per-layer context K/V cache (K [L,B,n_kv,cap,hd], V transposed [L,B,n_kv,hd,cap]) + lengths."""

    def __init__(self, shape, batch_cap: int, ctx_cap: int, device="cuda"):
        import torch
        if ctx_cap % 64:
            raise ValueError("ctx_cap must be a multiple of 64")
        dt = torch.bfloat16 if shape.dtype == "bf16" else torch.float32
        L, nkv, hd = shape.n_layers, shape.n_kv_heads, shape.head_dim
        self.k = torch.zeros((L, batch_cap, nkv, ctx_cap, hd), dtype=dt, device=device)
        self.v = torch.zeros((L, batch_cap, nkv, hd, ctx_cap), dtype=dt, device=device)
        self.ctx_len = torch.zeros(batch_cap, dtype=torch.int32, device=device)
        self.batch_cap, self.ctx_cap = batch_cap, ctx_cap
        self.c = DparaCtx(k=_ptr(self.k), v=_ptr(self.v), ctx_len=_ptr(self.ctx_len), batch_cap=batch_cap,
                          ctx_cap=ctx_cap)


class Workspace:
    def __init__(self, cfg: DparaConfig, batch: int, ctx_cap: int, device="cuda", target: bool = False):
        import torch
        self.nbytes = (dpara_target_workspace_bytes if target else dpara_workspace_bytes)(cfg, batch, ctx_cap)
        if self.nbytes == 0:
            raise DparaError(DPARA_E_INVALID, "invalid configuration for workspace sizing")
        self.buf = torch.empty(self.nbytes, dtype=torch.uint8, device=device)
        self.buf[:256].zero_()  # the header (status word, head flag) starts clear

    @property
    def ptr(self) -> int:
        return _ptr(self.buf)

    def status(self) -> int:
        import torch
        return int(self.buf[:4].view(torch.int32).item())

    def head_fallback(self) -> int:
        """Nonzero if the last select_and_head on this workspace needed the full head."""
        import torch
        return int(self.buf[4:8].view(torch.int32).item())


# ---------------------------------------------------------------- tensor-level calls
def ctx_append(d: DeviceDrafter, ctx: DeviceContext, feats, n_new, ws: Workspace, stream=None):
    """feats [B, n_max, H] (device, drafter dtype), n_new [B] int32 (device)."""
    B, n_max = int(feats.shape[0]), int(feats.shape[1])
    dpara_ctx_append(d.cfg, d.w, ctx.c, B, _ptr(feats), _ptr(n_new), n_max, ws.ptr, ws.nbytes, _stream(stream))


def backbone_all_boundaries(d: DeviceDrafter, ctx: DeviceContext, spine, reps, ws: Workspace, stream=None):
    dpara_backbone_all_boundaries(d.cfg, d.w, ctx.c, int(spine.shape[0]), _ptr(spine), _ptr(reps), ws.ptr,
                                  ws.nbytes, _stream(stream))


def backbone_trace(d: DeviceDrafter, ctx: DeviceContext, spine, reps, resid, ws: Workspace, stream=None):
    """backbone_all_boundaries that also writes resid [n_layers, B, (gamma+1)^2, H] float32: every
    row's residual stream after every layer."""
    _check(lib().dpara_backbone_trace(_ref(d.cfg), _ref(d.w), _ref(ctx.c), int(spine.shape[0]), _ptr(spine),
                                      _ptr(reps), _ptr(resid), ws.ptr, ws.nbytes, _stream(stream)))


def verify_greedy(d: DeviceDrafter, logits, spine, accept_len, bonus, target_argmax, ws: Workspace, stream=None):
    import torch
    ldt = DPARA_BF16 if logits.dtype == torch.bfloat16 else DPARA_F32
    dpara_verify_greedy(d.cfg, int(spine.shape[0]), _ptr(logits), ldt, _ptr(spine), _ptr(accept_len), _ptr(bonus),
                        _ptr(target_argmax), ws.ptr, ws.nbytes, _stream(stream))


def dpara_verify_greedy_noalloc(cfg, batch, target_logits, logits_dtype, spine, accept_len, bonus, target_argmax,
                                status, stream):
    _check(lib().dpara_verify_greedy_noalloc(_ref(cfg), batch, target_logits, logits_dtype, spine, accept_len, bonus,
                                             target_argmax, status, stream))


def verify_greedy_noalloc(d, logits, spine, accept_len, bonus, target_argmax=None, status=None, stream=None):
    """verify_greedy without a workspace (the library's static scratch); status: an int32 device
    tensor the DPARA_STATUS_* bits are OR-ed into, or None."""
    import torch
    ldt = DPARA_BF16 if logits.dtype == torch.bfloat16 else DPARA_F32
    dpara_verify_greedy_noalloc(d.cfg, int(spine.shape[0]), _ptr(logits), ldt, _ptr(spine), _ptr(accept_len),
                                _ptr(bonus), _ptr(target_argmax), _ptr(status), _stream(stream))


def select_and_head(d: DeviceDrafter, reps, accept_len, bonus, gathered, drafts, next_spine, margins,
                    ws: Workspace, stream=None):
    dpara_select_and_head(d.cfg, d.w, int(accept_len.shape[0]), _ptr(reps), _ptr(accept_len), _ptr(bonus),
                          _ptr(gathered), _ptr(drafts), _ptr(next_spine), _ptr(margins), ws.ptr, ws.nbytes,
                          _stream(stream))


def select_and_head_sampled(d: DeviceDrafter, reps, accept_len, bonus, gathered, drafts, next_spine, margins,
                            temperature: float, seed, scores, ws: Workspace, stream=None):
    """The sampled head: y_i ~ softmax(z_i / T) from the library's counter-based generator;
    scores [B, gamma, V] float32 (or None) receives z_i / T.  seed: an int, or a one-element
    int64 device tensor read when the kernels run."""
    seed_dev, seed = _seed_args(seed)
    _check(lib().dpara_select_and_head_sampled(_ref(d.cfg), _ref(d.w), int(accept_len.shape[0]), _ptr(reps),
                                               _ptr(accept_len), _ptr(bonus), _ptr(gathered), _ptr(drafts),
                                               _ptr(next_spine), _ptr(margins), float(temperature), seed,
                                               seed_dev, _ptr(scores), ws.ptr, ws.nbytes, _stream(stream)))


def _seed_args(seed):
    """(seed_dev pointer, host seed) for an int or a one-element int64 device tensor."""
    if isinstance(seed, int):
        return 0, seed & 0xFFFFFFFFFFFFFFFF
    assert seed.numel() == 1 and seed.element_size() == 8 and seed.is_cuda
    return _ptr(seed), 0


def verify_sampled(d: DeviceDrafter, logits, scores, spine, temperature: float, seed, accept_len, bonus,
                   ws: Workspace, stream=None):
    """Speculative-sampling verification: logits [B, gamma+1, V] (bf16 or float32), scores
    [B, gamma, V] float32 (the drafts' tempered scores), spine [B, gamma+1] int32; seed as for
    select_and_head_sampled."""
    import torch
    seed_dev, seed = _seed_args(seed)
    ldt = DPARA_BF16 if logits.dtype == torch.bfloat16 else DPARA_F32
    _check(lib().dpara_verify_sampled(_ref(d.cfg), int(spine.shape[0]), _ptr(logits), ldt, _ptr(scores),
                                      _ptr(spine), float(temperature), seed, seed_dev, _ptr(accept_len), _ptr(bonus),
                                      ws.ptr, ws.nbytes, _stream(stream)))


def branch_candidates_buffer(d: DeviceDrafter, batch: int, device="cuda"):
    """A device buffer for dpara_branch_candidates (256-byte aligned)."""
    import torch
    n = dpara_branch_candidates_bytes(d.cfg, batch)
    return torch.zeros(n, dtype=torch.uint8, device=device)


def branch_candidates(d: DeviceDrafter, reps, cand, ws: Workspace, stream=None):
    dpara_branch_candidates(d.cfg, d.w, int(reps.shape[0]), _ptr(reps), _ptr(cand), ws.ptr, ws.nbytes,
                            _stream(stream))


def select_and_head_cand(d: DeviceDrafter, reps, cand, accept_len, bonus, gathered, drafts, next_spine, margins,
                         ws: Workspace, stream=None):
    dpara_select_and_head_cand(d.cfg, d.w, int(accept_len.shape[0]), _ptr(reps), _ptr(cand), _ptr(accept_len),
                               _ptr(bonus), _ptr(gathered), _ptr(drafts), _ptr(next_spine), _ptr(margins), ws.ptr,
                               ws.nbytes, _stream(stream))


def dpara_fuse_workspace_bytes(cfg, n_rows: int, n_feat: int) -> int:
    return int(lib().dpara_fuse_workspace_bytes(ctypes.byref(cfg), n_rows, n_feat))


def dpara_fuse_features(cfg, fw, n_rows, hidden, feats, ws, ws_bytes, stream):
    _check(lib().dpara_fuse_features(_ref(cfg), _ref(fw), n_rows, hidden, feats, ws, ws_bytes, stream))


class DeviceFusion:
    """Feature-fusion weights resident in HBM (fc [H, n_feat*H], norm gain [H]) plus the
    C struct that points at them."""

    def __init__(self, shape, weights: dict | None, n_feat: int, device="cuda", seed: int = 7):
        import torch
        from . import synth
        self.shape = shape
        self.cfg = make_config(shape)
        mdt = torch.bfloat16 if shape.dtype == "bf16" else torch.float32
        if weights is None:  # generated on device (timing only)
            self.fc = synth.device_normal_(torch.empty((shape.hidden, n_feat * shape.hidden), dtype=mdt,
                                                       device=device), seed, 0.02)
            self.norm = torch.ones(shape.hidden, dtype=torch.float32, device=device)
        else:
            self.fc = torch.from_numpy(np.ascontiguousarray(weights["fc"])).to(device=device, dtype=mdt)
            self.norm = torch.from_numpy(np.ascontiguousarray(weights["fc_norm"])).to(device=device,
                                                                                       dtype=torch.float32)
        self.n_feat = n_feat
        self.w = DparaFusionWeights(fc=_ptr(self.fc), norm=_ptr(self.norm), n_feat=n_feat)


def fuse_features(f: DeviceFusion, hidden, feats, ws, stream=None):
    """hidden [n, n_feat*H] -> feats [n, H] (cfg dtype, on device); ws a uint8 device tensor
    of at least dpara_fuse_workspace_bytes bytes."""
    n = int(hidden.shape[0])
    dpara_fuse_features(f.cfg, f.w, n, _ptr(hidden), _ptr(feats), _ptr(ws), int(ws.numel()), _stream(stream))


def target_forward_hidden(t: DeviceTarget, ctx: DeviceContext, block, logits, feat_layers, hidden, ws: Workspace,
                          stream=None):
    """target_forward that also writes hidden [B, gamma+1, n_feat, H] (bf16): the block rows'
    residual stream after each layer of feat_layers."""
    import torch
    ldt = DPARA_BF16 if logits.dtype == torch.bfloat16 else DPARA_F32
    fl = (ctypes.c_int32 * len(feat_layers))(*[int(x) for x in feat_layers])
    _check(lib().dpara_target_forward_hidden(_ref(t.cfg), _ref(t.w), _ref(ctx.c), int(block.shape[0]), _ptr(block),
                                             _ptr(logits), ldt, fl, len(feat_layers), _ptr(hidden), ws.ptr,
                                             ws.nbytes, _stream(stream)))


def target_forward(t: DeviceTarget, ctx: DeviceContext, block, logits, ws: Workspace, stream=None):
    """block [B, gamma+1] int32, logits [B, gamma+1, V] (bf16 or float32) on device."""
    import torch
    ldt = DPARA_BF16 if logits.dtype == torch.bfloat16 else DPARA_F32
    dpara_target_forward(t.cfg, t.w, ctx.c, int(block.shape[0]), _ptr(block), _ptr(logits), ldt, ws.ptr,
                         ws.nbytes, _stream(stream))
