"""GPU parity: the HIP path (through the C ABI) against the CPU oracle on the same seeded inputs.

Bars: accepted lengths, bonus, target argmax and gathered rows bit-exact;
representations within 1e-5 (float32 model) or 2e-2 (bf16 model) max-abs; draft
ids exact wherever the oracle's top1 - top2 margin of z_i exceeds 1e-2, checked
teacher-forced (the oracle's step i is fed the GPU's y_{i-1}).

Deep bf16 drafters (5 layers at 4096/5120 width): every layer is held to the stated
2e-2 bar on its own, teacher-forced (test_layerwise_teacher_forced: the oracle's layer
on the GPU's own input residual, every row of the sampled requests).  End to end,
float32 accumulation alone (instead of the oracle's float64) flips a fraction of the
bf16 roundings and the flips compound with depth: running the oracle's own GEMMs and
attention in float32 moves it from itself, at the Qwen3-8B shape, by up to 3.7e-2
max-abs on request 0 of the batch-1 round (99.99th percentile 2.9e-2, median 5e-3) and
by 3.4e-2 on the sampled rows of the batch-16 round, while one full-width layer stays
at 1.1e-2.  The end-to-end comparison of the 5-layer configurations is therefore a
documented envelope, not the parity bar: max-abs <= 5e-2, 99.99th percentile <=
3.5e-2, median <= 1e-2; single-layer and small configurations keep 2e-2 end to end.
"""
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import dpara_oracle as O  # noqa: E402
from paper_2609_27396_amd import synth  # noqa: E402

pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-5, "bf16": 2e-2}
DEEP = {"max": 5e-2, "q9999": 3.5e-2, "median": 1e-2}
MARGIN = 1e-2


def check_reps(shape, err_arrays, tag):
    """Apply the bar for `shape` to a list of |gpu - oracle| arrays; returns max."""
    d = np.concatenate([np.ravel(e) for e in err_arrays])
    mx, q, med = float(d.max()), float(np.quantile(d, 0.9999)), float(np.median(d))
    _say(f"{tag}: |reps-oracle| max {mx:.3e} q99.99 {q:.3e} median {med:.2e}")
    if shape.dtype == "f32":
        assert mx <= TOL["f32"]
    elif shape.n_layers > 1 and shape.hidden >= 4096:
        assert mx <= DEEP["max"] and q <= DEEP["q9999"] and med <= DEEP["median"]
    else:
        assert mx <= TOL["bf16"]
    return mx


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _harness():
    from paper_2609_27396_amd.harness import DeviceRound
    return DeviceRound


def check_verify(ri, dr):
    acc, bon, tg = dr.accept.cpu().numpy(), dr.bonus.cpu().numpy(), dr.targmax.cpu().numpy()
    for b in range(dr.B):
        r, bonus, g = O.verify_greedy(ri.target_logits[b], ri.spine[b])
        assert acc[b] == r and bon[b] == bonus, (b, acc[b], r, bon[b], bonus)
        np.testing.assert_array_equal(tg[b], g)
        assert r == ri.accept_planted[b] and bonus == ri.bonus_planted[b]


def check_head(shape, w, dr, mode, b):
    """Teacher-forced check of the AR head on the GPU's own gathered rows."""
    gathered = dr.gathered[b].cpu().numpy()
    r = int(dr.accept[b].item())
    np.testing.assert_array_equal(gathered, dr.reps[b, r].cpu().numpy())   # bit-exact gather
    drafts = dr.drafts[b].cpu().numpy()
    nxt = dr.next_spine[b].cpu().numpy()
    bonus = int(dr.bonus[b].item())
    assert nxt[0] == bonus
    np.testing.assert_array_equal(nxt[1:], drafts)
    ell = O.base_logits(w, gathered, mode)
    y_prev, skipped = bonus, 0
    gm = dr.margins[b].cpu().numpy()
    for i in range(shape.gamma):
        y, m, _ = O.head_step(w, ell[i], y_prev, mode)
        if m > MARGIN:
            assert drafts[i] == y, (b, i, drafts[i], y, m)
            assert abs(gm[i] - m) < 1e-3 + 1e-3 * abs(m)
        else:
            skipped += 1
        y_prev = int(drafts[i])
    return skipped


def run_full(wl: synth.Workload, weights, ri, ctx_cap=None):
    DeviceRound = _harness()
    dr = DeviceRound(wl.shape, weights, ri, ctx_cap=ctx_cap)
    dr.backbone()
    dr.verify()
    dr.head()
    torch.cuda.synchronize()
    assert dr.status() == 0
    return dr


# ----------------------------------------------------------------------------- tiny fp32 config
def test_tiny_round_parity():
    wl = synth.WORKLOADS["tiny"]
    _say("case tiny fp32 round", wl.description)
    w = synth.make_weights(wl.shape, seed=wl.seed_w, gain_jitter=0.1)
    ri = synth.make_round(wl)
    dr = run_full(wl, w, ri)
    check_verify(ri, dr)
    for b in range(wl.batch):
        ref = O.backbone_all_boundaries(wl.shape, w, ri.ctx_feats[b], ri.spine[b], "f32")["reps"]
        check_reps(wl.shape, [np.abs(dr.reps[b].cpu().numpy() - ref)], "tiny")
        check_head(wl.shape, w, dr, "f32", b)


# ----------------------------------------------------------------------------- small bf16 shapes
SMALL_CASES = {
    # several GEMM tiles with ragged M/N tails, hd 128, qk-norm, ragged contexts incl. an empty one
    "h256_hd128_g5": (synth.DrafterShape(n_layers=2, hidden=256, n_q_heads=4, n_kv_heads=2, head_dim=128, ffn=576,
                                         vocab=4000, gamma=5, ar_rank=64, qk_norm=True, dtype="bf16"),
                      [0, 77, 300]),
    # head_dim 64, no qk-norm, GQA 4:1
    "h512_hd64_g3": (synth.DrafterShape(n_layers=1, hidden=512, n_q_heads=8, n_kv_heads=2, head_dim=64, ffn=640,
                                        vocab=1000, gamma=3, ar_rank=128, qk_norm=False, dtype="bf16"),
                     [64, 129]),
    # the shortest draft: two boundaries
    "h256_g1": (synth.DrafterShape(n_layers=1, hidden=256, n_q_heads=4, n_kv_heads=2, head_dim=64, ffn=512,
                                   vocab=2000, gamma=1, ar_rank=64, qk_norm=True, dtype="bf16"),
                [0, 50, 7]),
    # the longest draft the library takes: 64 boundaries, 4096 block rows per request
    "h256_g63": (synth.DrafterShape(n_layers=1, hidden=256, n_q_heads=4, n_kv_heads=2, head_dim=64, ffn=512,
                                    vocab=2000, gamma=63, ar_rank=64, qk_norm=True, dtype="bf16"),
                 [100, 3]),
    # mixed context lengths with ties and empty contexts: attention orders the requests longest
    # context first (ties by index)
    "h256_g3_ties": (synth.DrafterShape(n_layers=1, hidden=256, n_q_heads=4, n_kv_heads=2, head_dim=64, ffn=512,
                                        vocab=1500, gamma=3, ar_rank=64, qk_norm=True, dtype="bf16"),
                     [90, 90, 5, 200, 90, 0, 200, 7, 7, 150, 0, 33]),
    # more than 64 requests: attention keeps the batch order
    "h256_g2_b70": (synth.DrafterShape(n_layers=1, hidden=256, n_q_heads=4, n_kv_heads=2, head_dim=64, ffn=512,
                                       vocab=1000, gamma=2, ar_rank=64, qk_norm=True, dtype="bf16"),
                    [(37 * i) % 180 for i in range(70)]),
    # float32 model with several tiles, hd 128
    "f32_h256_g7": (synth.DrafterShape(n_layers=2, hidden=256, n_q_heads=4, n_kv_heads=1, head_dim=128, ffn=320,
                                       vocab=3001, gamma=7, ar_rank=64, qk_norm=True, dtype="f32"),
                    [33, 150]),
}


@pytest.mark.parametrize("case", sorted(SMALL_CASES))
def test_small_parity(case):
    shape, ctx = SMALL_CASES[case]
    _say("case", case)
    wl = synth.Workload(case, shape, batch=len(ctx), ctx_min=0, ctx_max=0, p_reject=0.3, seed_in=7,
                        logits_dtype="bf16" if shape.dtype == "bf16" else "f32")
    w = synth.make_weights(shape, seed=3, gain_jitter=0.1, ar_e_std=1.0)
    ri = synth.make_round(wl, ctx_lens=ctx)
    dr = run_full(wl, w, ri)
    check_verify(ri, dr)
    mode = shape.dtype
    errs, skipped = [], 0
    for b in range(wl.batch):
        ref = O.backbone_all_boundaries(shape, w, ri.ctx_feats[b], ri.spine[b], mode)["reps"]
        errs.append(np.abs(dr.reps[b].cpu().numpy() - ref))
        skipped += check_head(shape, w, dr, mode, b)
    _say(case, "head steps skipped (margin<=1e-2):", skipped)
    check_reps(shape, errs, case)


HEAD_SHAPE = synth.DrafterShape(n_layers=1, hidden=256, n_q_heads=4, n_kv_heads=2, head_dim=64, ffn=512,
                                vocab=5000, gamma=6, ar_rank=128, qk_norm=True, dtype="bf16")


@pytest.mark.parametrize("regime", ["pruned", "full"])
def test_head_pruned_bound_and_fallback(regime):
    """The exact bound-pruned head proves every step when the correction W.E(y) is small
    next to the logit gaps (small ar_W), and hands the call to the full head when it cannot
    (large ar_W and ar_E: the bound max|W_v| |e| swamps every gap); both give the oracle's
    drafts and margins."""
    shape = HEAD_SHAPE
    _say("case head", regime)
    wl = synth.Workload("head_" + regime, shape, batch=3, ctx_min=0, ctx_max=0, p_reject=0.3, seed_in=11,
                        logits_dtype="bf16")
    big = regime == "full"
    w = synth.make_weights(shape, seed=5, gain_jitter=0.1, ar_w_std=2.0 if big else 0.005,
                           ar_e_std=1.0 if big else 0.02)
    ri = synth.make_round(wl, ctx_lens=[40, 0, 100])
    dr = run_full(wl, w, ri)
    check_verify(ri, dr)
    fb = dr.head_fallback()
    _say(regime, "fallback flag", fb)
    assert (fb != 0) if big else (fb == 0)
    skipped = sum(check_head(shape, w, dr, "bf16", b) for b in range(wl.batch))
    assert skipped < wl.batch * shape.gamma // 2


@pytest.mark.parametrize("regime", ["pruned", "full"])
def test_prepared_head_norm_gives_the_same_head(regime):
    """With the weights' max |W_v|^2 prepared once (dpara_head_prepare), the greedy and the
    sampled head give the same drafts, next block, margins, scores and fallback flag, bit for
    bit, as the per-call pass over W, whether every step is proven or the full head runs."""
    shape = HEAD_SHAPE
    big = regime == "full"
    wl = synth.Workload("hp", shape, batch=3, ctx_min=0, ctx_max=0, p_reject=0.3, seed_in=12)
    w = synth.make_weights(shape, seed=5, gain_jitter=0.1, ar_w_std=2.0 if big else 0.005,
                           ar_e_std=1.0 if big else 0.02)
    ri = synth.make_round(wl, ctx_lens=[20, 0, 90])
    dr = _harness()(shape, w, ri)
    dr.backbone()
    dr.verify()
    scores = torch.empty((3, shape.gamma, shape.vocab), dtype=torch.float32, device="cuda")
    outs = ("drafts", "next_spine", "margins")

    def run():
        dr.head()
        torch.cuda.synchronize()
        greedy = {k: getattr(dr, k).clone() for k in outs}
        gflag = dr.head_fallback()
        dr.head_sampled(1.0, 77, scores)
        torch.cuda.synchronize()
        sampled = {k: getattr(dr, k).clone() for k in outs}
        return greedy, gflag, sampled, dr.head_fallback(), scores.clone()

    ref = run()
    dr.d.prepare_head(dr.ws)
    assert float(dr.d.norm2.item()) == float((w["ar_W"].astype(np.float32) ** 2).sum(1).max()) or \
        abs(float(dr.d.norm2.item()) / float((w["ar_W"].astype(np.float64) ** 2).sum(1).max()) - 1) < 1e-6
    got = run()
    dr.d.unprepare_head()
    for r_, g_ in ((ref[0], got[0]), (ref[2], got[2])):
        for k in outs:
            assert torch.equal(r_[k], g_[k]), k
    assert (ref[1], ref[3]) == (got[1], got[3])
    assert (ref[1] != 0) == big
    assert torch.equal(ref[4], got[4])
    assert dr.status() == 0


@pytest.mark.parametrize("regime", ["pruned", "full"])
def test_head_from_branch_candidates(regime):
    """The off-serial-path head variant: candidates of every branch row computed after the
    backbone, then the serial step from the accepted branch's candidates.  Drafts, margins,
    next spine and gathered rows agree with the plain select + head where both prove every
    step, and with the oracle either way (the large-W regime takes the fallback)."""
    shape = HEAD_SHAPE
    _say("case head from candidates", regime)
    wl = synth.Workload("headc_" + regime, shape, batch=3, ctx_min=0, ctx_max=0, p_reject=0.3, seed_in=13,
                        logits_dtype="bf16")
    big = regime == "full"
    w = synth.make_weights(shape, seed=6, gain_jitter=0.1, ar_w_std=2.0 if big else 0.005,
                           ar_e_std=1.0 if big else 0.02)
    ri = synth.make_round(wl, ctx_lens=[70, 5, 0])
    dr = run_full(wl, w, ri)
    plain = {k: getattr(dr, k).clone() for k in ("drafts", "next_spine", "margins", "gathered")}
    fb_plain = dr.head_fallback()
    for k in ("drafts", "next_spine", "margins", "gathered"):
        getattr(dr, k).fill_(-7)
    dr.candidates()
    dr.head_cand()
    torch.cuda.synchronize()
    assert dr.status() == 0
    fb = dr.head_fallback()
    _say(regime, "fallback flags plain / candidates", fb_plain, fb)
    assert (fb != 0) if big else (fb == 0)
    assert torch.equal(dr.gathered, plain["gathered"])
    if fb == 0 and fb_plain == 0:
        for k in ("drafts", "next_spine", "margins"):
            assert torch.equal(getattr(dr, k), plain[k]), k
    for b in range(wl.batch):
        check_head(shape, w, dr, "bf16", b)


# Nine layers: the context append projects K|V for at most eight layers per GEMM, so this
# takes two layer groups (8 + 1), each layer with its own W_k, W_v and k-norm gains.
L9_SHAPE = synth.DrafterShape(n_layers=9, hidden=256, n_q_heads=4, n_kv_heads=2, head_dim=128, ffn=512,
                              vocab=3000, gamma=4, ar_rank=64, qk_norm=True, dtype="bf16")


def test_append_layer_groups_against_oracle():
    """Every layer's cached K and V after the prefill (context append over nine layers, two
    projection groups) is that layer's own incremental projection of the cached features:
    the oracle's context K/V within one bf16 rounding.  (The nine-layer reps themselves are
    not held to the single-layer bar: bf16 rounding flips compound through depth.)"""
    shape, ctx = L9_SHAPE, [45, 130]
    wl = synth.Workload("l9", shape, batch=len(ctx), ctx_min=0, ctx_max=0, p_reject=0.3, seed_in=7)
    w = synth.make_weights(shape, seed=3, gain_jitter=0.1)
    ri = synth.make_round(wl, ctx_lens=ctx)
    DeviceRound = _harness()
    dr = DeviceRound(shape, w, ri)
    torch.cuda.synchronize()
    assert dr.status() == 0
    rnd = O.Rounding("bf16")
    worst = 0.0
    for b, n in enumerate(ctx):
        for l in range(shape.n_layers):
            k_ref, v_ref = O.context_kv(shape, w, l, ri.ctx_feats[b], 0, rnd)
            k = dr.ctx.k[l, b, :, :n].float().cpu().numpy().transpose(1, 0, 2)     # [n, n_kv, hd]
            v = dr.ctx.v[l, b, :, :, :n].float().cpu().numpy().transpose(2, 0, 1)  # [n, n_kv, hd]
            for got, ref in ((k, k_ref), (v, v_ref)):
                err = np.abs(got - ref)
                worst = max(worst, float((err / (np.abs(ref) + 1e-4)).max()))
                assert np.all(err <= 2.0 ** -7 * np.abs(ref) + 1e-4), (b, l)
    _say("l9 append: worst relative |cache - oracle|", worst)


@pytest.mark.parametrize("case", ["h256_hd128_g5", "l9"])
def test_append_equivalence_and_determinism(case):
    shape = L9_SHAPE if case == "l9" else SMALL_CASES[case][0]
    wl = synth.Workload("app", shape, batch=2, ctx_min=0, ctx_max=0, p_reject=0.3, seed_in=9)
    w = synth.make_weights(shape, seed=4)
    ri = synth.make_round(wl, ctx_lens=[120, 61])
    DeviceRound = _harness()
    a = DeviceRound(shape, w, ri, ctx_cap=256)
    # b: prefill all but the last k rows, then append them
    k = np.array([6, 3], np.int32)
    ri_short = synth.RoundInputs(ctx_lens=ri.ctx_lens - k, ctx_feats=[f[:-kk] for f, kk in zip(ri.ctx_feats, k)],
                                 spine=ri.spine, accept_planted=ri.accept_planted, bonus_planted=ri.bonus_planted,
                                 target_logits=ri.target_logits, new_feats=ri.new_feats)
    bdr = DeviceRound(shape, w, ri_short, ctx_cap=256, drafter=a.d)
    tail = np.zeros((2, 6, shape.hidden), np.float32)
    for i, (f, kk) in enumerate(zip(ri.ctx_feats, k)):
        tail[i, :kk] = f[-kk:]
    bdr.append(torch.from_numpy(k).cuda(), torch.from_numpy(tail).cuda().to(torch.bfloat16))
    torch.cuda.synchronize()
    assert torch.equal(a.ctx.ctx_len, bdr.ctx.ctx_len)
    for b in range(2):
        n = int(ri.ctx_lens[b])
        assert torch.equal(a.ctx.k[:, b, :, :n], bdr.ctx.k[:, b, :, :n])
        assert torch.equal(a.ctx.v[:, b, :, :, :n], bdr.ctx.v[:, b, :, :, :n])
    a.backbone()
    r1 = a.reps.clone()
    a.backbone()
    bdr.backbone()
    torch.cuda.synchronize()
    assert torch.equal(r1, a.reps)          # determinism
    assert torch.equal(a.reps, bdr.reps)    # same cache => same result
    assert a.status() == 0


def test_device_status_flags_and_clamping():
    shape, _ = SMALL_CASES["h512_hd64_g3"]
    wl = synth.Workload("st", shape, batch=2, ctx_min=0, ctx_max=0, p_reject=0.3, seed_in=11)
    w = synth.make_weights(shape, seed=5)
    ri = synth.make_round(wl, ctx_lens=[10, 20])
    DeviceRound = _harness()
    dr = DeviceRound(shape, w, ri, ctx_cap=64)
    from paper_2609_27396_amd import dpara as D
    dr.spine[0, 1] = shape.vocab + 5           # out-of-range draft id: clamped, flagged
    dr.backbone()
    dr.verify()
    assert dr.status() & D.STATUS_TOKEN_RANGE
    assert int(dr.accept[0]) == 0              # an invalid draft never matches
    D.dpara_clear_status(dr.ws.ptr, D._stream(None))
    assert dr.status() == 0
    dr.accept[1] = shape.gamma + 3             # verdict out of range: clamped, flagged
    dr.head()
    assert dr.status() & D.STATUS_VERDICT_RANGE
    D.dpara_clear_status(dr.ws.ptr, D._stream(None))
    n_new = torch.tensor([60, 2], dtype=torch.int32, device="cuda")  # 10 + 60 > 64
    feats = torch.zeros((2, 60, shape.hidden), dtype=torch.bfloat16, device="cuda")
    dr.append(n_new, feats)
    assert dr.status() & D.STATUS_CTX_FULL
    assert dr.ctx.ctx_len.cpu().tolist() == [64, 22]
    D.dpara_clear_status(dr.ws.ptr, D._stream(None))
    dr.append(torch.tensor([-1, 99], dtype=torch.int32, device="cuda"), feats)
    assert dr.status() & D.STATUS_COUNT_RANGE
    assert dr.ctx.ctx_len.cpu().tolist() == [64, 64]


# ----------------------------------------------------------------------------- full-size configs
def _full_size(name, samples):
    wl = synth.WORKLOADS[name]
    _say("case", name, wl.description)
    w = synth.make_weights(wl.shape, seed=wl.seed_w)
    ri = synth.make_round(wl)
    dr = run_full(wl, w, ri)
    check_verify(ri, dr)
    errs, skipped = [], 0
    for b, branches in samples:
        for r in branches:
            one = O.backbone_single_boundary(wl.shape, w, ri.ctx_feats[b], ri.spine[b], r, "bf16")
            err = np.abs(dr.reps[b, r].cpu().numpy() - one["reps"])
            _say(f"{name} request {b} (ctx {ri.ctx_lens[b]}) branch {r}: max|reps-oracle| = {err.max():.3e}")
            errs.append(err)
        skipped += check_head(wl.shape, w, dr, "bf16", b)
    _say(name, "head steps skipped:", skipped)
    check_reps(wl.shape, errs, name)
    return dr, ri


def test_full_width_one_layer_qwen3_8b():
    """One Qwen3-8B-width layer, context 2048, gamma 16: every branch against the oracle's tree pass."""
    import dataclasses
    base = synth.WORKLOADS["qwen3_8b_b1"]
    shape = dataclasses.replace(base.shape, n_layers=1)
    wl = dataclasses.replace(base, name="qwen3_8b_1layer", shape=shape)
    _say("case qwen3_8b width, 1 layer, ctx 2048, gamma 16, all branches")
    w = synth.make_weights(shape, seed=wl.seed_w, gain_jitter=0.1)
    ri = synth.make_round(wl)
    dr = run_full(wl, w, ri)
    check_verify(ri, dr)
    ref = O.backbone_all_boundaries(shape, w, ri.ctx_feats[0], ri.spine[0], "bf16")["reps"]
    check_reps(shape, [np.abs(dr.reps[0].cpu().numpy() - ref)], "qwen3_8b_1layer")
    check_head(shape, w, dr, "bf16", 0)


def test_full_size_qwen3_8b_b1():
    """Every branch of the batch-1 request, end to end, against the oracle's tree pass."""
    wl = synth.WORKLOADS["qwen3_8b_b1"]
    _say("case qwen3_8b_b1 end to end, all branches")
    w = synth.make_weights(wl.shape, seed=wl.seed_w)
    ri = synth.make_round(wl)
    dr = run_full(wl, w, ri)
    check_verify(ri, dr)
    ref = O.backbone_all_boundaries(wl.shape, w, ri.ctx_feats[0], ri.spine[0], "bf16")["reps"]
    check_reps(wl.shape, [np.abs(dr.reps[0].cpu().numpy() - ref)], "qwen3_8b_b1 all branches")
    _say("qwen3_8b_b1 head steps skipped:", check_head(wl.shape, w, dr, "bf16", 0))


# Requests checked layer by layer (all (gamma+1)^2 rows of each, spine rows included).
LAYERWISE = {"qwen3_8b_b1": (0,), "qwen3_8b_b16": (0, 6, 11, 15), "qwen3_14b_b8": (0, 7)}


@pytest.mark.parametrize("name", sorted(LAYERWISE))
def test_layerwise_teacher_forced(name):
    """Each drafter layer of the full-size configurations on its own, teacher-forced: the oracle's
    layer_forward runs on the GPU's own residual stream entering that layer (every row of the
    request: spine and every branch's masks; the oracle's own context K/V and tree mask), and its
    output is compared with the GPU's residual after the layer.  The bar is the stated 2e-2
    max-abs on the hidden representation, i.e. the residual normalised to unit root mean square
    (the scale the next layer's norm and the final representations see).  The final layer's mask
    rows, normalised with the final gain, are the reps the backbone returns (float32 rounding of
    the norm apart)."""
    from paper_2609_27396_amd import dpara as D
    wl = synth.WORKLOADS[name]
    s = wl.shape
    _say("case layerwise", name, wl.description)
    w = synth.make_weights(s, seed=wl.seed_w)
    ri = synth.make_round(wl)
    dr = _harness()(s, w, ri)
    R, g, H, L = s.rows, s.gamma, s.hidden, s.n_layers
    resid = torch.empty((L, dr.B, R, H), dtype=torch.float32, device="cuda")
    D.backbone_trace(dr.d, dr.ctx, dr.spine, dr.reps, resid, dr.ws)
    reps_trace = dr.reps.clone()
    dr.backbone()
    torch.cuda.synchronize()
    assert dr.status() == 0
    assert torch.equal(reps_trace, dr.reps)   # tracing leaves the result unchanged
    rnd = O.Rounding("bf16")
    vis = O.tree_visibility(g)
    worst = 0.0
    for b in LAYERWISE[name]:
        n_b = int(ri.ctx_lens[b])
        pos = O.row_positions(g, n_b)
        x_in = np.empty((R, H), np.float64)
        for j in range(g + 1):
            x_in[j] = w["embed"][int(ri.spine[b, j])]
        x_in[g + 1:] = w["mask_emb"][None, :]
        for l in range(L):
            ck, cv = O.context_kv(s, w, l, ri.ctx_feats[b], 0, rnd)
            x_ref = O.layer_forward(s, w, l, x_in, pos, ck, cv, vis, rnd)
            x_gpu = resid[l, b].cpu().numpy().astype(np.float64)
            h_ref, h_gpu = O.rmsnorm(x_ref, 1.0, s.rms_eps), O.rmsnorm(x_gpu, 1.0, s.rms_eps)
            e = np.abs(h_gpu - h_ref)
            rms = float(np.sqrt(np.mean(x_ref ** 2)))
            _say(f"{name} request {b} (ctx {n_b}) layer {l}: max|h-oracle| {e.max():.3e} (spine rows "
                 f"{e[:g + 1].max():.3e}), q99.99 {np.quantile(e, 0.9999):.3e}, residual rms {rms:.3f}, "
                 f"max|x-oracle|/rms {np.abs(x_gpu - x_ref).max() / rms:.3e}")
            worst = max(worst, float(e.max()))
            assert e.max() <= TOL["bf16"], (name, b, l)
            x_in = x_gpu
        reps = O.rmsnorm(x_in[g + 1:], w["final_norm"], s.rms_eps).reshape(g + 1, g, H)
        np.testing.assert_allclose(dr.reps[b].cpu().numpy(), reps, rtol=1e-5, atol=1e-5)
    _say(name, "layerwise worst max-abs", worst)


def test_full_size_qwen3_8b_b16():
    wl = synth.WORKLOADS["qwen3_8b_b16"]
    ri = synth.make_round(wl)
    samples = [(b, [int(ri.accept_planted[b])]) for b in (0, 7, 15)]
    _full_size("qwen3_8b_b16", samples)


def test_full_size_qwen3_14b_b8():
    """Qwen3-14B-shaped drafter (hidden 5120, 40/8 heads, FFN 17408), batch 8 at context 8192:
    the accepted branch of the first and last request against the oracle, head teacher-forced."""
    wl = synth.WORKLOADS["qwen3_14b_b8"]
    ri = synth.make_round(wl)
    samples = [(b, [int(ri.accept_planted[b])]) for b in (0, wl.batch - 1)]
    _full_size("qwen3_14b_b8", samples)


# ----------------------------------------------------------------------------- target verification forward
TARGET_SMALL = synth.DrafterShape(n_layers=2, hidden=256, n_q_heads=4, n_kv_heads=2, head_dim=128, ffn=512,
                                  vocab=3001, gamma=5, ar_rank=64, qk_norm=True, dtype="bf16")


def _target_setup(ctx_lens, cap=256, seed=7):
    from paper_2609_27396_amd import dpara as D
    from paper_2609_27396_amd.harness import upload_cache
    s = TARGET_SMALL
    w = synth.make_target_weights(s, seed=seed, gain_jitter=0.1)
    k, v = synth.make_target_cache(s, ctx_lens, seed=seed + 1)
    block = np.random.default_rng(seed).integers(0, s.vocab, (len(ctx_lens), s.gamma + 1)).astype(np.int32)
    t = D.DeviceTarget(s, w)
    ctx = D.DeviceContext(s, len(ctx_lens), cap)
    upload_cache(ctx, k, v, ctx_lens, torch.bfloat16)
    ws = D.Workspace(t.cfg, len(ctx_lens), cap, target=True)
    return s, w, k, v, block, t, ctx, ws


def test_target_forward_parity():
    from paper_2609_27396_amd import dpara as D
    ctx_lens = [0, 50, 200]
    _say("case target forward: 2 layers, 256 wide, block 6, contexts", ctx_lens)
    s, w, k, v, block, t, ctx, ws = _target_setup(ctx_lens)
    blk = torch.from_numpy(block).cuda()
    lf = torch.empty((len(ctx_lens), s.gamma + 1, s.vocab), dtype=torch.float32, device="cuda")
    lb = torch.empty_like(lf, dtype=torch.bfloat16)
    D.target_forward(t, ctx, blk, lf, ws)
    D.target_forward(t, ctx, blk, lb, ws)
    torch.cuda.synchronize()
    errs, skipped = [], 0
    for b, n in enumerate(ctx_lens):
        ref = O.target_forward(s, w, [k[l][b] for l in range(s.n_layers)], [v[l][b] for l in range(s.n_layers)],
                               block[b], "bf16")
        got = lf[b].cpu().numpy()
        errs.append(np.abs(got - ref))
        for j in range(s.gamma + 1):
            y, m = O.argmax_margin(ref[j])
            if m > MARGIN:
                assert int(np.argmax(got[j])) == y
            else:
                skipped += 1
    d = np.concatenate([e.ravel() for e in errs])
    _say(f"target logits |gpu-oracle| max {d.max():.3e} median {np.median(d):.2e}, argmax rows skipped {skipped}")
    assert d.max() <= TOL["bf16"]
    # bf16 logits are the float32 logits rounded once
    np.testing.assert_allclose(lb.float().cpu().numpy(), lf.cpu().numpy(), rtol=2 ** -8, atol=0)
    # emitting hidden states leaves the logits bit for bit as they were; the hidden states
    # are the oracle's residual stream after those layers, within the bf16 bar
    fl = [1, 0]
    hid = torch.empty((len(ctx_lens), s.gamma + 1, len(fl), s.hidden), dtype=torch.bfloat16, device="cuda")
    lh = torch.empty_like(lf)
    D.target_forward_hidden(t, ctx, blk, lh, fl, hid, ws)
    torch.cuda.synchronize()
    assert torch.equal(lh, lf)
    for b in range(len(ctx_lens)):
        _, th = O.target_forward(s, w, [k[l][b] for l in range(s.n_layers)], [v[l][b] for l in range(s.n_layers)],
                                 block[b], "bf16", fl)
        got = hid[b].float().cpu().numpy()
        assert np.all(np.abs(got - th) <= 2.0 ** -8 * np.abs(th) + TOL["bf16"]), b


def test_backbone_and_target_on_concurrent_streams():
    """The drafter backbone and the target forward on two streams at once give the same bits as
    run alone, and those are the oracle's: reps within the bf16 bar of the oracle's tree pass,
    target logits within the bar of the oracle's target forward (argmax equal where the margin
    exceeds 1e-2)."""
    from paper_2609_27396_amd import dpara as D
    DeviceRound = _harness()
    shape, _ = SMALL_CASES["h256_hd128_g5"]
    wl = synth.Workload("cc", shape, batch=3, ctx_min=0, ctx_max=0, p_reject=0.3, seed_in=13)
    wd = synth.make_weights(shape, seed=14)
    ri = synth.make_round(wl, ctx_lens=[40, 0, 170])
    dr = DeviceRound(shape, wd, ri)
    s, w, k, v, block, t, ctx, ws = _target_setup([10, 120, 33], seed=21)
    blk = torch.from_numpy(block).cuda()
    l1 = torch.empty((3, s.gamma + 1, s.vocab), dtype=torch.bfloat16, device="cuda")
    l2 = torch.empty_like(l1)
    dr.backbone()
    D.target_forward(t, ctx, blk, l1, ws)
    torch.cuda.synchronize()
    reps1 = dr.reps.clone()
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    for _ in range(3):
        dr.reps.zero_()
        torch.cuda.synchronize()
        with torch.cuda.stream(s1):
            dr.backbone(stream=s1)
        with torch.cuda.stream(s2):
            D.target_forward(t, ctx, blk, l2, ws, stream=s2)
        torch.cuda.synchronize()
        assert torch.equal(reps1, dr.reps)
        assert torch.equal(l1, l2)
    errs = []
    for b in range(3):
        ref = O.backbone_all_boundaries(shape, wd, ri.ctx_feats[b], ri.spine[b], "bf16")["reps"]
        errs.append(np.abs(dr.reps[b].cpu().numpy() - ref))
        tl = O.target_forward(s, w, [k[l][b] for l in range(s.n_layers)], [v[l][b] for l in range(s.n_layers)],
                              block[b], "bf16")
        got = l2[b].float().cpu().numpy()
        assert np.all(np.abs(got - tl) <= 2.0 ** -8 * np.abs(tl) + TOL["bf16"]), b
        for j in range(s.gamma + 1):
            y, m = O.argmax_margin(tl[j])
            if m > MARGIN + 2.0 ** -7 * np.abs(tl[j]).max():  # the logits here are bf16
                assert int(np.argmax(got[j])) == y, (b, j)
    check_reps(shape, errs, "concurrent streams")


def test_verification_beside_backbone_on_one_workspace():
    """Greedy and sampled verification on a second stream, concurrent with the backbone on the
    same workspace (context capacity 512, so the backbone splits its attention over more key
    ranges than a 64-capacity plan would): every output equals the sequential run's bit for bit."""
    from paper_2609_27396_amd import dpara as D
    DeviceRound = _harness()
    shape, _ = SMALL_CASES["h256_hd128_g5"]
    wl = synth.Workload("vb", shape, batch=3, ctx_min=0, ctx_max=0, p_reject=0.3, seed_in=15)
    wd = synth.make_weights(shape, seed=16)
    ri = synth.make_round(wl, ctx_lens=[300, 17, 450])
    dr = DeviceRound(shape, wd, ri, ctx_cap=512)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(3)
    scores = torch.randn((3, shape.gamma, shape.vocab), generator=gen, device="cuda", dtype=torch.float32)
    acc2, bon2 = torch.empty_like(dr.accept), torch.empty_like(dr.bonus)

    def verify_both(stream=None):
        dr.verify(stream=stream)
        D.verify_sampled(dr.d, dr.logits, scores, dr.spine, 1.0, 99, acc2, bon2, dr.ws, stream)

    dr.backbone()
    verify_both()
    torch.cuda.synchronize()
    ref = [t.clone() for t in (dr.reps, dr.accept, dr.bonus, dr.targmax, acc2, bon2)]
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    for _ in range(3):
        for t in (dr.reps, dr.accept, dr.bonus, dr.targmax, acc2, bon2):
            t.zero_()
        torch.cuda.synchronize()
        with torch.cuda.stream(s1):
            dr.backbone(stream=s1)
        with torch.cuda.stream(s2):
            verify_both(stream=s2)
        torch.cuda.synchronize()
        for a_, b_ in zip(ref, (dr.reps, dr.accept, dr.bonus, dr.targmax, acc2, bon2)):
            assert torch.equal(a_, b_)
    assert dr.status() == 0


# ----------------------------------------------------------------------------- HIP graph of a round
@pytest.mark.parametrize("case", ["h256_hd128_g5", "qwen3_8b_b1", "h256_hd128_g5_sampled", "qwen3_8b_b1_sampled"])
def test_round_graph_replays(case):
    """One steady-state round (context rewind, append of the accepted rows' features,
    all-boundary backbone, greedy verify, select + head) captured into a HIP graph: every
    replay, with eager work that overwrites the outputs and synchronisations between the
    replays, gives the eager round's results bit for bit (the library takes all scratch from
    the caller's workspace and launches only kernels on the caller's stream).  The sampled
    cases capture the sampling variant's verification and head instead, with the seed read
    from device memory: replays alternate two seeds written there between replays, and each
    replay matches the eager round with that seed (scores the head writes included)."""
    sampled = case.endswith("_sampled")
    case = case[:-len("_sampled")] if sampled else case
    if case == "qwen3_8b_b1":
        wl = synth.WORKLOADS[case]
        w = synth.make_weights(wl.shape, seed=wl.seed_w)
        ri = synth.make_round(wl)
    else:
        shape, ctx = SMALL_CASES[case]
        wl = synth.Workload(case, shape, batch=len(ctx), ctx_min=0, ctx_max=0, p_reject=0.3, seed_in=7,
                            logits_dtype="bf16")
        w = synth.make_weights(shape, seed=3, gain_jitter=0.1)
        ri = synth.make_round(wl, ctx_lens=ctx)
    DeviceRound = _harness()
    dr = DeviceRound(wl.shape, w, ri)
    B = wl.batch
    n_new_h = ri.accept_planted.astype(np.int32) + 1
    n_new = torch.from_numpy(n_new_h).cuda()
    base_len = torch.from_numpy((ri.ctx_lens - n_new_h).astype(np.int32)).cuda()
    outs = ("reps", "accept", "bonus", "targmax", "gathered", "drafts", "next_spine", "margins")
    if sampled:
        g_, V_ = wl.shape.gamma, wl.shape.vocab
        gen = torch.Generator(device="cuda")
        gen.manual_seed(5)
        dr.scores_in = torch.randn((B, g_, V_), generator=gen, device="cuda", dtype=torch.float32)
        dr.scores_out = torch.empty((B, g_, V_), dtype=torch.float32, device="cuda")
        dr.targmax.zero_()  # not written by the sampled verification
        outs = ("reps", "accept", "bonus", "gathered", "drafts", "next_spine", "margins", "scores_out")
        seeds = (1234, 987654321987)
        seed_t = torch.tensor([seeds[0]], dtype=torch.int64, device="cuda")

    def step():
        dr.ctx.ctx_len[:B].copy_(base_len)
        dr.append(n_new)
        dr.backbone()
        if sampled:
            dr.verify_sampled(dr.scores_in, 1.0, seed_t)
            dr.head_sampled(1.0, seed_t, dr.scores_out)
        else:
            dr.verify()
            dr.head()

    refs = []
    for sd in (seeds if sampled else (None,)):
        if sampled:
            seed_t.fill_(sd)
        step()  # eager (also the first call of every launcher outside the capture)
        torch.cuda.synchronize()
        assert dr.status() == 0
        refs.append({k: getattr(dr, k).clone() for k in outs})
    if sampled:
        assert not torch.equal(refs[0]["drafts"], refs[1]["drafts"])  # the seed reaches the draws
    ref = refs[-1]
    ref_len = dr.ctx.ctx_len.clone()
    ref_k, ref_v = dr.ctx.k.clone(), dr.ctx.v.clone()
    g = torch.cuda.CUDAGraph()
    cs = torch.cuda.Stream()
    cs.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(cs):
        with torch.cuda.graph(g, stream=cs):
            step()
    torch.cuda.synchronize()
    for rep in range(4):
        if sampled:
            seed_t.fill_(seeds[rep % 2])
            ref = refs[rep % 2]
        for k in outs:  # eager work between the replays
            t = getattr(dr, k)
            t.fill_(-7 if t.dtype == torch.int32 else float("nan"))
        dr.ctx.ctx_len.fill_(0)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for k in outs:
            assert torch.equal(getattr(dr, k), ref[k]), (rep, k)
        assert torch.equal(dr.ctx.ctx_len, ref_len)
        assert torch.equal(dr.ctx.k, ref_k) and torch.equal(dr.ctx.v, ref_v)
        assert dr.status() == 0
    _say(case, "sampled" if sampled else "greedy", "graph replays identical to the eager round: 4")
    # the last replay against the oracle: the context is the rewound prefix plus the appended rows
    mode, errs = wl.shape.dtype, []
    for b in range(B):
        n0 = int(ri.ctx_lens[b]) - int(n_new_h[b])
        feats = np.concatenate([ri.ctx_feats[b][:n0], ri.new_feats[b][:int(n_new_h[b])]])
        ref = O.backbone_all_boundaries(wl.shape, w, feats, ri.spine[b], mode)["reps"]
        errs.append(np.abs(dr.reps[b].cpu().numpy() - ref))
    check_reps(wl.shape, errs, case + " graph replay")
    if sampled:
        from test_gpu_sampling import ACC_MARGIN, BONUS_MARGIN, _check_head_sampled
        seed, s_in = seeds[3 % 2], dr.scores_in.cpu().numpy()
        for b in range(B):
            r, bonus, info = O.verify_sampled(ri.target_logits[b], s_in[b], ri.spine[b], 1.0, seed, b)
            if np.abs(info["accept_margins"]).min() > ACC_MARGIN:
                assert int(dr.accept[b]) == r, (b, int(dr.accept[b]), r)
                if info["bonus_margin"] > BONUS_MARGIN:
                    assert int(dr.bonus[b]) == bonus, b
        compared = _check_head_sampled(wl.shape, w, dr, dr.scores_out, 1.0, seed, mode)
        assert compared >= B * wl.shape.gamma - 2
    else:
        check_verify(ri, dr)
        for b in range(B):
            check_head(wl.shape, w, dr, mode, b)



def test_full_round_graph_two_streams():
    """Single-GPU colocation as one HIP graph (Section 4.3.2 and Appendix D: both forward passes
    on two streams of one GPU and the head captured together).  Captured: a fork onto two streams
    (the target's verification forward of the block on one; the drafter's context rewind, append
    and all-boundary backbone on the other), the join, then the greedy verdict kernel and select +
    head, whose inputs are device buffers.  Every replay, with eager work clobbering the outputs in
    between, equals the eager round bit for bit; the last replay matches the oracle (target logits,
    verdict from them, reps over the rewound prefix plus the appended rows, head teacher-forced).
    The host reads the verdict and drafts after the replay (the acceptance bookkeeping stays
    outside the graph)."""
    from paper_2609_27396_amd import dpara as D
    from paper_2609_27396_amd.harness import upload_cache
    sd, st_ = LOOP_DRAFTER, LOOP_TARGET
    ctx_lens, B, g = [40, 0, 170], 3, LOOP_DRAFTER.gamma
    wd = synth.make_weights(sd, seed=51, gain_jitter=0.1, ar_e_std=1.0)
    wt = synth.make_target_weights(st_, seed=52, gain_jitter=0.1)
    wl = synth.Workload("fr", sd, batch=B, ctx_min=0, ctx_max=0, p_reject=0.3, seed_in=53)
    ri = synth.make_round(wl, ctx_lens=ctx_lens)
    dr = _harness()(sd, wd, ri, ctx_cap=256)
    tk, tv = synth.make_target_cache(st_, ctx_lens, seed=54)
    t = D.DeviceTarget(st_, wt)
    tctx = D.DeviceContext(st_, B, 256)
    upload_cache(tctx, tk, tv, ctx_lens, torch.bfloat16)
    tws = D.Workspace(t.cfg, B, 256, target=True)
    n_new_h = ri.accept_planted.astype(np.int32) + 1
    n_new = torch.from_numpy(n_new_h).cuda()
    base_len = torch.from_numpy((ri.ctx_lens - n_new_h).astype(np.int32)).cuda()
    s_v, s_d = torch.cuda.Stream(), torch.cuda.Stream()

    def round_():
        cur = torch.cuda.current_stream()
        s_v.wait_stream(cur)
        s_d.wait_stream(cur)
        with torch.cuda.stream(s_d):
            dr.ctx.ctx_len[:B].copy_(base_len)
            dr.append(n_new, stream=s_d)
            dr.backbone(stream=s_d)
        with torch.cuda.stream(s_v):
            D.target_forward(t, tctx, dr.spine, dr.logits, tws, stream=s_v)
        cur.wait_stream(s_d)
        cur.wait_stream(s_v)
        dr.verify()
        dr.head()

    outs = ("logits", "reps", "accept", "bonus", "targmax", "gathered", "drafts", "next_spine", "margins")
    round_()
    torch.cuda.synchronize()
    assert dr.status() == 0
    ref = {k: getattr(dr, k).clone() for k in outs}
    ref_k, ref_v = dr.ctx.k.clone(), dr.ctx.v.clone()
    graph = torch.cuda.CUDAGraph()
    cs = torch.cuda.Stream()
    cs.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(cs):
        with torch.cuda.graph(graph, stream=cs):
            round_()
    torch.cuda.synchronize()
    for rep in range(4):
        for k in outs:
            x = getattr(dr, k)
            x.fill_(-7 if x.dtype == torch.int32 else float("nan"))
        dr.ctx.ctx_len.fill_(0)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for k in outs:
            assert torch.equal(getattr(dr, k), ref[k]), (rep, k)
        assert torch.equal(dr.ctx.k, ref_k) and torch.equal(dr.ctx.v, ref_v)
        assert dr.status() == 0
    lg = dr.logits.float().cpu().numpy()
    acc, bon, tg = dr.accept.cpu().numpy(), dr.bonus.cpu().numpy(), dr.targmax.cpu().numpy()
    errs, compared = [], 0
    for b in range(B):
        tl = O.target_forward(st_, wt, [tk[l][b] for l in range(st_.n_layers)],
                              [tv[l][b] for l in range(st_.n_layers)], ri.spine[b], "bf16")
        assert np.all(np.abs(lg[b] - tl) <= 2.0 ** -8 * np.abs(tl) + TOL["bf16"]), b
        r, bonus, gg = O.verify_greedy(lg[b], ri.spine[b])     # the verdict of the GPU's logits: exact
        assert (int(acc[b]), int(bon[b])) == (r, bonus) and np.array_equal(tg[b], gg), b
        r_o, bonus_o, _ = O.verify_greedy(tl, ri.spine[b])    # and the oracle's, where its margins allow
        if min(O.argmax_margin(tl[j])[1] for j in range(r_o + 1)) > MARGIN + 2.0 ** -7 * np.abs(tl).max():
            assert (r, bonus) == (r_o, bonus_o), b
            compared += 1
        n0 = int(ri.ctx_lens[b]) - int(n_new_h[b])
        feats = np.concatenate([ri.ctx_feats[b][:n0], ri.new_feats[b][:int(n_new_h[b])]])
        rep_ref = O.backbone_all_boundaries(sd, wd, feats, ri.spine[b], "bf16")["reps"]
        errs.append(np.abs(dr.reps[b].cpu().numpy() - rep_ref))
        check_head(sd, wd, dr, "bf16", b)
    check_reps(sd, errs, "full-round graph replay")
    _say("full-round graph: 4 replays identical to the eager round; verdicts compared with the oracle's:",
         compared, "accepted", acc.tolist())


# ----------------------------------------------------------------------------- feature fusion
FUSE_CASES = {
    # rows: one, a round's worth, several 64-row tiles with a ragged tail, above 320 rows
    "h256_bf16": (synth.DrafterShape(n_layers=1, hidden=256, n_q_heads=4, n_kv_heads=2, head_dim=64, ffn=512,
                                     vocab=1000, gamma=4, ar_rank=64, qk_norm=True, dtype="bf16"),
                  [1, 17, 333, 700]),
    "h256_f32": (synth.DrafterShape(n_layers=1, hidden=256, n_q_heads=4, n_kv_heads=2, head_dim=64, ffn=512,
                                    vocab=1000, gamma=4, ar_rank=64, qk_norm=True, dtype="f32"),
                 [5, 90]),
    # Qwen3-8B width: a round at b=1, a 2048-row prefill (one pass of under a round of large
    # tiles) and a prefill that spans two 4096-row passes
    "qwen3_8b": (synth.QWEN3_8B, [17, 2048, 4100]),
}


@pytest.mark.parametrize("case", sorted(FUSE_CASES))
def test_fuse_features_parity(case):
    """Fused features f = RMSNorm(fc [h_1; h_2; h_3]) * g against the oracle: bf16 results
    within one bf16 rounding (float32 projection either side), float32 within 1e-5; the
    4100-row case checks rows on both sides of the 4096-row pass boundary."""
    from paper_2609_27396_amd import dpara as D
    shape, row_counts = FUSE_CASES[case]
    n_feat = 3
    wf = synth.make_fusion_weights(shape, n_feat=n_feat, seed=11, gain_jitter=0.1)
    fus = D.DeviceFusion(shape, wf, n_feat)
    mdt = torch.bfloat16 if shape.dtype == "bf16" else torch.float32
    worst = 0.0
    for n in row_counts:
        hid = synth.make_target_hidden(shape, n, n_feat=n_feat, seed=12 + n)
        hd = torch.from_numpy(hid).to(device="cuda", dtype=mdt)
        out = torch.empty((n, shape.hidden), dtype=mdt, device="cuda")
        ws = torch.empty(D.dpara_fuse_workspace_bytes(fus.cfg, n, n_feat), dtype=torch.uint8, device="cuda")
        D.fuse_features(fus, hd, out, ws)
        torch.cuda.synchronize()
        rows = np.arange(n) if n <= 1000 else np.unique(np.r_[0:40, 1000:1010, 4080:4100, n - 5:n])
        rows = rows[rows < n]
        ref = O.fuse_features(shape, wf, hid[rows], shape.dtype)
        got = out.float().cpu().numpy()[rows]
        err = np.abs(got - ref)
        if shape.dtype == "bf16":
            # one bf16 rounding, plus the float32 summation error of a 3H-term projection
            # (about 1e-5 after the norm at H = 4096) where a value sits near zero
            bad = err > 2.0 ** -7 * np.abs(ref) + 1e-4
        else:
            bad = err > 1e-5 * np.maximum(np.abs(ref), 1.0)
        worst = max(worst, float((err / (np.abs(ref) + 1e-6)).max()))
        if bad.any():
            i = np.argwhere(bad)[0]
            _say("fusion mismatch", n, tuple(i), float(got[tuple(i)]), float(ref[tuple(i)]))
        assert not bad.any(), (n, int(bad.sum()))
    _say(case, "fusion: worst relative |gpu - oracle|", worst)


# ----------------------------------------------------------------------------- Algorithm 1 iterated
LOOP_DRAFTER = synth.DrafterShape(n_layers=2, hidden=256, n_q_heads=4, n_kv_heads=2, head_dim=128, ffn=512,
                                  vocab=3001, gamma=5, ar_rank=64, qk_norm=True, dtype="bf16")
LOOP_TARGET = synth.DrafterShape(n_layers=4, hidden=256, n_q_heads=4, n_kv_heads=2, head_dim=128, ffn=512,
                                 vocab=3001, gamma=5, ar_rank=64, qk_norm=True, dtype="bf16")
FEAT_LAYERS = [0, 1, 3]
LOOP_PLANT = [0, 3, 5]   # leading drafts of each round's block replaced by the target's own greedy chain


def _greedy_chain(st_, wt, tk, tv, b, t0, k):
    """t_0 followed by k tokens of the oracle target's greedy continuation (causal, so the
    block's verdict accepts at least those k drafts)."""
    blk = [int(t0)]
    for _ in range(k):
        lg = O.target_forward(st_, wt, [tk[l][b] for l in range(st_.n_layers)],
                              [tv[l][b] for l in range(st_.n_layers)], np.array(blk, np.int32), "bf16")
        blk.append(int(np.argmax(lg[-1])))
    return blk


def test_iterated_rounds_with_fused_target_features():
    """Algorithm 1 iterated over three rounds on random weights.  Each round the target
    forwards the block and emits its hidden states after layers 0, 1 and 3; greedy verify;
    the drafter's all-boundary backbone and select + head; the hidden states of the block are
    fused and the rows of t_0..t_r are appended to the drafter's cache (C <- [C, C_new]).
    The loop is driven by the oracle: every round's block is the oracle's next spine (with
    a planted number of leading drafts replaced by the target's greedy chain, so the accepted
    length varies from 0 to gamma) and the append count is the oracle's r + 1; the GPU's
    hidden states, logits, verdict, reps, drafts and fused rows are checked against the
    oracle's, wherever the oracle's argmax margins make them unique.  Both contexts grow by the
    oracle's fused rows (the GPU's own fused rows are checked against them separately), so every
    round's reps are held to the single-round bar on identical inputs.  The target's own cache
    stays fixed."""
    from paper_2609_27396_amd import dpara as D
    from paper_2609_27396_amd.harness import upload_cache
    sd, st_ = LOOP_DRAFTER, LOOP_TARGET
    ctx_lens, B, g, H = [30, 90], 2, LOOP_DRAFTER.gamma, LOOP_DRAFTER.hidden
    nf = len(FEAT_LAYERS)
    wd = synth.make_weights(sd, seed=31, gain_jitter=0.1, ar_e_std=1.0)
    wt = synth.make_target_weights(st_, seed=32, gain_jitter=0.1)
    wf = synth.make_fusion_weights(sd, n_feat=nf, seed=33, gain_jitter=0.1)
    wl = synth.Workload("loop", sd, batch=B, ctx_min=0, ctx_max=0, p_reject=0.3, seed_in=34)
    ri = synth.make_round(wl, ctx_lens=ctx_lens)
    dr = _harness()(sd, wd, ri, ctx_cap=256)
    tk, tv = synth.make_target_cache(st_, ctx_lens, seed=35)
    t = D.DeviceTarget(st_, wt)
    tctx = D.DeviceContext(st_, B, 256)
    upload_cache(tctx, tk, tv, ctx_lens, torch.bfloat16)
    tws = D.Workspace(t.cfg, B, 256, target=True)
    fus = D.DeviceFusion(sd, wf, nf)
    fws = torch.empty(D.dpara_fuse_workspace_bytes(fus.cfg, B * (g + 1), nf), dtype=torch.uint8, device="cuda")
    hid = torch.empty((B, g + 1, nf, H), dtype=torch.bfloat16, device="cuda")
    fused = torch.empty((B, g + 1, H), dtype=torch.bfloat16, device="cuda")
    feats = [np.asarray(f, np.float32) for f in ri.ctx_feats]  # the oracle's drafter context
    spine = ri.spine.astype(np.int32).copy()
    worst = {"hidden": 0.0, "logits": 0.0, "reps": 0.0, "fused": 0.0}
    compared = {"verdicts": 0, "drafts": 0, "n_new": []}
    for rnd in range(len(LOOP_PLANT)):
        for b in range(B):
            chain = _greedy_chain(st_, wt, tk, tv, b, spine[b, 0], LOOP_PLANT[rnd])
            spine[b, :len(chain)] = chain
        _say(f"round {rnd}: planted {LOOP_PLANT[rnd]}, spine {spine.tolist()}")
        dr.spine.copy_(torch.from_numpy(spine))
        D.target_forward_hidden(t, tctx, dr.spine, dr.logits, FEAT_LAYERS, hid, tws)
        dr.backbone()
        dr.verify()
        dr.head()
        D.fuse_features(fus, hid.view(B * (g + 1), nf * H), fused.view(B * (g + 1), H), fws)
        torch.cuda.synchronize()
        assert dr.status() == 0
        acc, bonus = dr.accept.cpu().numpy(), dr.bonus.cpu().numpy()
        drafts = dr.drafts.cpu().numpy()
        logits_h = dr.logits.float().cpu().numpy()
        hid_h, fused_h = hid.float().cpu().numpy(), fused.float().cpu().numpy()
        nxt, n_new = np.zeros_like(spine), np.zeros(B, np.int32)
        f_app = np.zeros((B, g + 1, H), np.float32)
        for b in range(B):
            tl, th = O.target_forward(st_, wt, [tk[l][b] for l in range(st_.n_layers)],
                                      [tv[l][b] for l in range(st_.n_layers)], spine[b], "bf16", FEAT_LAYERS)
            # the GPU's hidden states and logits are rounded once to bf16 from float32 values
            # within the bf16 bar of the oracle's
            e = np.abs(hid_h[b] - th)
            worst["hidden"] = max(worst["hidden"], float(e.max()))
            assert np.all(e <= 2.0 ** -8 * np.abs(th) + TOL["bf16"]), (rnd, b)
            e = np.abs(logits_h[b] - tl)
            worst["logits"] = max(worst["logits"], float(e.max()))
            assert np.all(e <= 2.0 ** -8 * np.abs(tl) + TOL["bf16"]), (rnd, b)
            r_ref, bonus_ref, _ = O.verify_greedy(tl, spine[b])
            assert r_ref >= LOOP_PLANT[rnd]
            if min(O.argmax_margin(tl[j])[1] for j in range(r_ref + 1)) > MARGIN:
                assert (int(acc[b]), int(bonus[b])) == (r_ref, bonus_ref), (rnd, b)
                compared["verdicts"] += 1
            ref = O.backbone_all_boundaries(sd, wd, feats[b], spine[b], "bf16")["reps"]
            e = np.abs(dr.reps[b].cpu().numpy() - ref)
            worst["reps"] = max(worst["reps"], float(e.max()))
            assert e.max() <= TOL["bf16"], (rnd, b)
            check_head(sd, wd, dr, "bf16", b)
            hd = O.select_and_head(sd, wd, ref, r_ref, bonus_ref, "bf16")
            if int(acc[b]) == r_ref:
                for i in range(g):           # the oracle's own chain, up to its first near-tie
                    if hd["margins"][i] <= MARGIN:
                        break
                    assert int(drafts[b, i]) == int(hd["drafts"][i]), (rnd, b, i)
                    compared["drafts"] += 1
            # C_new: the fused target features of t_0..t_r.  The GPU fuses its own hidden
            # states, which already sit within the bf16 bar of the oracle's, so the fused rows
            # are held to that end-to-end bar (the fusion kernel's own bar, on identical
            # inputs, is checked by the fusion parity test)
            k = r_ref + 1
            f_ref = O.fuse_features(sd, wf, th[:k].reshape(k, nf * H), "bf16")
            e = np.abs(fused_h[b, :k] - f_ref)
            worst["fused"] = max(worst["fused"], float(e.max()))
            assert np.all(e <= 2.0 ** -7 * np.abs(f_ref) + TOL["bf16"]), (rnd, b)
            feats[b] = np.concatenate([feats[b], f_ref.astype(np.float32)])
            f_app[b, :k] = f_ref
            nxt[b], n_new[b] = hd["next_spine"], k
        before = dr.ctx.ctx_len[:B].clone()
        nn = torch.from_numpy(n_new).cuda()
        dr.append(nn, torch.from_numpy(f_app).cuda().to(torch.bfloat16))   # the oracle's rows, bf16-valued
        torch.cuda.synchronize()
        assert torch.equal(dr.ctx.ctx_len[:B], before + nn)
        assert dr.status() == 0
        compared["n_new"].append(n_new.tolist())
        spine = nxt
    _say("iterated rounds: worst |gpu - oracle|", worst, "compared", compared)
    assert compared["verdicts"] >= 4
