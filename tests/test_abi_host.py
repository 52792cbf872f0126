"""Host-side checks of the C ABI: exports, workspace sizing and argument validation.

These run without a GPU: every call here fails validation before any HIP call."""
import ctypes
import dataclasses
import os
import re

import pytest

from paper_2609_27396_amd import dpara as D
from paper_2609_27396_amd import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _header_functions():
    txt = open(os.path.join(ROOT, "include", "dpara.h")).read()
    return sorted(set(re.findall(r"^\s*(?:size_t|int|int32_t|const char\s*\*)\s*(dpara_\w+)\s*\(", txt, re.M)))


def test_library_loads_and_exports_every_declared_symbol():
    names = _header_functions()
    assert len(names) >= 8
    L = D.lib()
    for n in names:
        assert hasattr(L, n), n
    assert set(D.EXPORTS) == set(names)
    assert D.dpara_version() == 100


def test_workspace_bytes():
    cfg = D.make_config(synth.QWEN3_8B)
    a = D.dpara_workspace_bytes(cfg, 1, 2112)
    b = D.dpara_workspace_bytes(cfg, 16, 4160)
    assert 0 < a < b
    assert D.dpara_workspace_bytes(cfg, 1, 100) == 0        # ctx_cap not a multiple of 64
    assert D.dpara_workspace_bytes(cfg, 0, 2112) == 0
    bad = D.make_config(synth.shrink(synth.QWEN3_8B, head_dim=96))
    assert D.dpara_workspace_bytes(bad, 1, 2112) == 0
    bad = D.make_config(synth.shrink(synth.QWEN3_8B, gamma=64))
    assert D.dpara_workspace_bytes(bad, 1, 2112) == 0
    bad = D.make_config(synth.shrink(synth.QWEN3_8B, n_kv_heads=7))
    assert D.dpara_workspace_bytes(bad, 1, 2112) == 0


FAKE = 1 << 20  # a 16-byte aligned non-null address; never dereferenced (validation fails first)


def _fake_weights(shape):
    layers = (D.DparaLayerWeights * shape.n_layers)()
    for l in range(shape.n_layers):
        for f, _ in D.DparaLayerWeights._fields_:
            setattr(layers[l], f, FAKE)
    w = D.DparaWeights(embed=FAKE, mask_emb=FAKE, final_norm=FAKE, ar_E=FAKE, ar_W=FAKE,
                       layers=ctypes.cast(layers, ctypes.POINTER(D.DparaLayerWeights)))
    return w, layers


def _rc(fn, *args):
    return getattr(D.lib(), fn)(*args)


def test_validation_errors_without_gpu():
    s = synth.shrink(synth.QWEN3_8B, n_layers=2)
    cfg = D.make_config(s)
    w, _keep = _fake_weights(s)
    ctx = D.DparaCtx(k=FAKE, v=FAKE, ctx_len=FAKE, batch_cap=2, ctx_cap=2112)
    need = D.dpara_workspace_bytes(cfg, 2, 2112)
    R = ctypes.byref
    # workspace too small
    assert _rc("dpara_backbone_all_boundaries", R(cfg), R(w), R(ctx), 2, FAKE, FAKE, FAKE, need - 1, None) \
        == D.DPARA_E_WORKSPACE
    assert "needs" in D.dpara_last_error()
    # batch above the cache's batch capacity
    assert _rc("dpara_backbone_all_boundaries", R(cfg), R(w), R(ctx), 3, FAKE, FAKE, FAKE, need, None) \
        == D.DPARA_E_CAPACITY
    # null / misaligned pointers
    assert _rc("dpara_backbone_all_boundaries", R(cfg), R(w), R(ctx), 2, None, FAKE, FAKE, need, None) \
        == D.DPARA_E_INVALID
    assert _rc("dpara_backbone_all_boundaries", R(cfg), R(w), R(ctx), 2, FAKE, FAKE + 4, FAKE, need, None) \
        == D.DPARA_E_INVALID
    w.mask_emb = None
    assert _rc("dpara_backbone_all_boundaries", R(cfg), R(w), R(ctx), 2, FAKE, FAKE, FAKE, need, None) \
        == D.DPARA_E_INVALID
    assert "mask_emb" in D.dpara_last_error()
    # bad configuration
    bad = D.make_config(synth.shrink(s, gamma=0))
    assert _rc("dpara_backbone_all_boundaries", R(bad), R(w), R(ctx), 2, FAKE, FAKE, FAKE, need, None) \
        == D.DPARA_E_INVALID
    bad = D.make_config(s)
    bad.dtype = 7
    assert _rc("dpara_verify_greedy", R(bad), 1, FAKE, 0, FAKE, FAKE, FAKE, None, FAKE, need, None) \
        == D.DPARA_E_UNSUPPORTED
    # verify: unsupported logits dtype, null outputs
    assert _rc("dpara_verify_greedy", R(cfg), 1, FAKE, 5, FAKE, FAKE, FAKE, None, FAKE, need, None) \
        == D.DPARA_E_UNSUPPORTED
    assert _rc("dpara_verify_greedy", R(cfg), 1, FAKE, 1, FAKE, None, FAKE, None, FAKE, need, None) \
        == D.DPARA_E_INVALID
    # append: n_max < 1, ctx_cap not a multiple of 64
    assert _rc("dpara_ctx_append", R(cfg), R(w), R(ctx), 2, FAKE, FAKE, 0, FAKE, need, None) == D.DPARA_E_INVALID
    ctx_bad = D.DparaCtx(k=FAKE, v=FAKE, ctx_len=FAKE, batch_cap=2, ctx_cap=100)
    assert _rc("dpara_ctx_append", R(cfg), R(w), R(ctx_bad), 2, FAKE, FAKE, 4, FAKE, need, None) \
        == D.DPARA_E_INVALID
    # head: null drafts
    assert _rc("dpara_select_and_head", R(cfg), R(w), 1, FAKE, FAKE, FAKE, None, None, FAKE, None, FAKE, need,
               None) == D.DPARA_E_INVALID


def test_binding_raises_loudly_on_error():
    s = synth.TINY
    cfg = D.make_config(s)
    with pytest.raises(D.DparaError) as e:
        D.dpara_verify_greedy(cfg, 1, FAKE, 9, FAKE, FAKE, FAKE, None, FAKE, 1 << 20, None)
    assert e.value.code == D.DPARA_E_UNSUPPORTED


def test_fusion_validation_without_gpu():
    """dpara_fuse_features rejects bad arguments on the host, before any launch."""
    cfg = D.make_config(synth.QWEN3_8B)
    need = D.dpara_fuse_workspace_bytes(cfg, 17, 3)
    assert need > 0
    assert D.dpara_fuse_workspace_bytes(cfg, 4100, 3) > need
    assert D.dpara_fuse_workspace_bytes(cfg, 0, 3) == 0
    assert D.dpara_fuse_workspace_bytes(cfg, 17, 9) == 0
    fw = D.DparaFusionWeights(fc=FAKE, norm=FAKE, n_feat=3)
    R = ctypes.byref
    ws = 1 << 24  # 256-byte aligned, never dereferenced
    assert _rc("dpara_fuse_features", R(cfg), R(fw), 17, FAKE, FAKE, ws, need - 1, None) == D.DPARA_E_WORKSPACE
    assert _rc("dpara_fuse_features", R(cfg), R(fw), 0, FAKE, FAKE, ws, need, None) == D.DPARA_E_INVALID
    assert _rc("dpara_fuse_features", R(cfg), R(fw), 17, FAKE + 8, FAKE, ws, need, None) == D.DPARA_E_INVALID
    assert _rc("dpara_fuse_features", R(cfg), R(fw), 17, FAKE, FAKE, ws + 64, need, None) == D.DPARA_E_INVALID
    bad = D.DparaFusionWeights(fc=FAKE, norm=FAKE, n_feat=0)
    assert _rc("dpara_fuse_features", R(cfg), R(bad), 17, FAKE, FAKE, ws, need, None) == D.DPARA_E_INVALID
    assert "n_feat" in D.dpara_last_error()
    bad = D.DparaFusionWeights(fc=None, norm=FAKE, n_feat=3)
    assert _rc("dpara_fuse_features", R(cfg), R(bad), 17, FAKE, FAKE, ws, need, None) == D.DPARA_E_INVALID


def test_target_hidden_validation_without_gpu():
    """dpara_target_forward_hidden rejects a bad feature-layer list on the host, before any launch."""
    cfg = D.make_config(synth.QWEN3_8B)
    R = ctypes.byref
    fl = (ctypes.c_int32 * 9)(*range(9))
    args = lambda fl, n, hid: (R(cfg), None, None, 1, FAKE, FAKE, D.DPARA_BF16, fl, n, hid, FAKE, 1 << 20, None)
    assert _rc("dpara_target_forward_hidden", *args(fl, 9, FAKE)) == D.DPARA_E_INVALID
    assert "n_feat" in D.dpara_last_error()
    assert _rc("dpara_target_forward_hidden", *args(fl, -1, FAKE)) == D.DPARA_E_INVALID
    assert _rc("dpara_target_forward_hidden", *args(None, 3, FAKE)) == D.DPARA_E_INVALID
    assert _rc("dpara_target_forward_hidden", *args(fl, 3, None)) == D.DPARA_E_INVALID
    assert _rc("dpara_target_forward_hidden", *args(fl, 3, FAKE + 8)) == D.DPARA_E_INVALID
    out = (ctypes.c_int32 * 3)(0, cfg.n_layers - 1, cfg.n_layers)
    assert _rc("dpara_target_forward_hidden", *args(out, 3, FAKE)) == D.DPARA_E_INVALID
    assert "feat_layers[2]" in D.dpara_last_error()


def test_sampling_validation_without_gpu():
    """The sampled head and verification reject a non-positive or non-finite temperature and
    missing buffers on the host, before any launch."""
    shape = synth.QWEN3_8B
    cfg = D.make_config(shape)
    w, _layers = _fake_weights(shape)
    R = ctypes.byref
    ws, nb = FAKE, D.dpara_workspace_bytes(cfg, 1, 64)
    for t in (0.0, -1.0, float("inf"), float("nan"), 1e-45):
        rc = _rc("dpara_select_and_head_sampled", R(cfg), R(w), 1, FAKE, FAKE, FAKE, None, FAKE, FAKE, None,
                 t, 1, None, None, ws, nb, None)
        assert rc == D.DPARA_E_INVALID, t
        assert "temperature" in D.dpara_last_error()
        rc = _rc("dpara_verify_sampled", R(cfg), 1, FAKE, D.DPARA_BF16, FAKE, FAKE, t, 1, None, FAKE, FAKE, ws, nb,
                 None)
        assert rc == D.DPARA_E_INVALID, t
    assert _rc("dpara_verify_sampled", R(cfg), 1, FAKE, D.DPARA_BF16, None, FAKE, 1.0, 1, None, FAKE, FAKE, ws, nb,
               None) == D.DPARA_E_INVALID
    assert "draft_scores" in D.dpara_last_error()
    assert _rc("dpara_verify_sampled", R(cfg), 1, FAKE, 7, FAKE, FAKE, 1.0, 1, None, FAKE, FAKE, ws, nb,
               None) == D.DPARA_E_UNSUPPORTED
    assert _rc("dpara_verify_sampled", R(cfg), 1, FAKE, D.DPARA_BF16, FAKE, FAKE, 1.0, 1, None, FAKE, FAKE, ws, 1024,
               None) == D.DPARA_E_WORKSPACE
    # the sampled head also needs the perturbed-logit and E-row regions at the end of the plan
    assert _rc("dpara_select_and_head_sampled", R(cfg), R(w), 1, FAKE, FAKE, FAKE, None, FAKE, FAKE, None,
               1.0, 1, None, None, ws, nb - 1, None) == D.DPARA_E_WORKSPACE


def test_head_prepare_validation_without_gpu():
    """dpara_head_prepare rejects a missing output, a missing or small workspace and an
    unsupported rank on the host, before any launch."""
    shape = synth.QWEN3_8B
    cfg = D.make_config(shape)
    w, _layers = _fake_weights(shape)
    R = ctypes.byref
    nb = D.dpara_workspace_bytes(cfg, 1, 64)
    assert _rc("dpara_head_prepare", R(cfg), R(w), None, FAKE, nb, None) == D.DPARA_E_INVALID
    assert "norm2_max" in D.dpara_last_error()
    assert _rc("dpara_head_prepare", R(cfg), R(w), FAKE, None, nb, None) == D.DPARA_E_INVALID
    assert _rc("dpara_head_prepare", R(cfg), R(w), FAKE, FAKE, 1024, None) == D.DPARA_E_WORKSPACE
    bad = D.make_config(synth.DrafterShape(n_layers=1, hidden=256, n_q_heads=2, n_kv_heads=1, head_dim=128,
                                           ffn=512, vocab=1000, gamma=4, ar_rank=32, qk_norm=True, dtype="bf16"))
    assert _rc("dpara_head_prepare", R(bad), R(w), FAKE, FAKE, nb, None) in (D.DPARA_E_INVALID,
                                                                           D.DPARA_E_UNSUPPORTED)
    assert "ar_rank" in D.dpara_last_error()


def test_candidates_prepare_validation_without_gpu():
    """dpara_candidates_prepare rejects a missing output, a missing, misaligned or small
    workspace and a float32 drafter on the host, before any launch."""
    shape = synth.QWEN3_8B
    cfg = D.make_config(shape)
    w, _layers = _fake_weights(shape)
    R = ctypes.byref
    nb = D.dpara_workspace_bytes(cfg, 1, 64)
    assert _rc("dpara_candidates_prepare", R(cfg), R(w), None, FAKE, nb, None) == D.DPARA_E_INVALID
    assert "embed_norm2_max" in D.dpara_last_error()
    assert _rc("dpara_candidates_prepare", R(cfg), R(w), FAKE, None, nb, None) == D.DPARA_E_INVALID
    assert _rc("dpara_candidates_prepare", R(cfg), R(w), FAKE, FAKE + 16, nb, None) == D.DPARA_E_INVALID
    assert _rc("dpara_candidates_prepare", R(cfg), R(w), FAKE, FAKE, 1024, None) == D.DPARA_E_WORKSPACE
    f32 = D.make_config(dataclasses.replace(shape, dtype="f32"))
    assert _rc("dpara_candidates_prepare", R(f32), R(w), FAKE, FAKE, nb, None) == D.DPARA_E_UNSUPPORTED


def test_trace_and_noalloc_validation_without_gpu():
    """dpara_backbone_trace needs its residual buffer; dpara_verify_greedy_noalloc rejects calls
    whose partials exceed its static scratch (1 MiB: at the Qwen3 vocabulary and gamma 16,
    batch 202 fits and 203 does not) and bad arguments, all before any launch."""
    s = synth.shrink(synth.QWEN3_8B, n_layers=2)
    cfg = D.make_config(s)
    w, _keep = _fake_weights(s)
    ctx = D.DparaCtx(k=FAKE, v=FAKE, ctx_len=FAKE, batch_cap=2, ctx_cap=2112)
    need = D.dpara_workspace_bytes(cfg, 2, 2112)
    R = ctypes.byref
    assert _rc("dpara_backbone_trace", R(cfg), R(w), R(ctx), 2, FAKE, FAKE, None, FAKE, need, None) \
        == D.DPARA_E_INVALID
    assert "resid" in D.dpara_last_error()
    assert _rc("dpara_backbone_trace", R(cfg), R(w), R(ctx), 2, FAKE, FAKE, FAKE + 4, FAKE, need, None) \
        == D.DPARA_E_INVALID
    assert _rc("dpara_backbone_trace", R(cfg), R(w), R(ctx), 2, FAKE, FAKE, FAKE, FAKE, need - 1, None) \
        == D.DPARA_E_WORKSPACE
    nv = "dpara_verify_greedy_noalloc"
    assert _rc(nv, R(cfg), 203, FAKE, 1, FAKE, FAKE, FAKE, None, None, None) == D.DPARA_E_WORKSPACE
    assert "1048576" in D.dpara_last_error()
    assert _rc(nv, R(cfg), 0, FAKE, 1, FAKE, FAKE, FAKE, None, None, None) == D.DPARA_E_INVALID
    assert _rc(nv, R(cfg), 1, FAKE, 5, FAKE, FAKE, FAKE, None, None, None) == D.DPARA_E_UNSUPPORTED
    assert _rc(nv, R(cfg), 1, FAKE, 1, FAKE, FAKE, None, None, None, None) == D.DPARA_E_INVALID
    assert _rc(nv, R(cfg), 1, FAKE, 1, FAKE, FAKE, FAKE, None, FAKE + 2, None) == D.DPARA_E_INVALID
    with pytest.raises(D.DparaError) as e:
        D.dpara_verify_greedy_noalloc(cfg, 203, FAKE, 1, FAKE, FAKE, FAKE, None, None, None)
    assert e.value.code == D.DPARA_E_WORKSPACE
