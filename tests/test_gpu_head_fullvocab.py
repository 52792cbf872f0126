"""The AR head at the Qwen3 vocabulary (151936 entries, draft length 16, rank 256), against the
oracle, through the C ABI.

The bound-pruned steps prove every step at the full-size shapes, so the parity tests of whole
rounds never reach the full head there.  The first cases make the pruned bound fail on purpose
(a large head matrix W and token embedding E: max_v |W_v| |E[y]| swamps every logit gap), so
that every call hands over to the full head: the single-launch head (one workgroup per CU, its
step exchange and bounded wait) at batch 1, 2 and 16, and the per-step kernels at batch 20.  Greedy
drafts are checked teacher-forced (the oracle's step i is fed the GPU's y_{i-1}) wherever the
oracle's top1 - top2 margin exceeds 1e-2; sampled draws likewise, with the tempered scores
within 1e-3 + 1e-3 |s|.  The last cases run the off-serial-path head (candidates of every
branch row ranked by the rows' bf16 hi part, then rescored) at the default weight scales, where
the steps are proven, against the plain head bit for bit and against the oracle, at batch 1, 2,
4, 9, 13 and 16 (each batch up to 4 takes its own LM-head tile); with the embedding's max row norm
prepared, the plain head over more than 128 gathered rows takes the same ranking over the
accepted rows, and gives the same bits (also through its fallback to the full head).  The head
reads only the gathered rows, the tied embedding and E, W, so the representations here are
synthetic N(0, 1) rows rather than a backbone's output."""
import dataclasses

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import dpara_oracle as O  # noqa: E402
from paper_2609_27396_amd import synth  # noqa: E402

pytestmark = pytest.mark.gpu

MARGIN = 1e-2
# only the embedding, E and W matter to the head; one narrow layer keeps the upload small
SHAPE = dataclasses.replace(synth.QWEN3_8B, n_layers=1, ffn=256)
_CACHE = {}


def _say(*a):
    print(*a, flush=True)


def _setup(regime="full"):
    """Weights (host and device, once per module and regime): "full" has a head bound no step
    can pass, "pruned" the default scales, where the bound proves the steps."""
    if regime not in _CACHE:
        from paper_2609_27396_amd import dpara as D
        _CACHE.clear()  # one regime's 151936-row matrices at a time
        kw = dict(ar_w_std=2.0, ar_e_std=1.0) if regime == "full" else {}
        w = synth.make_weights(SHAPE, seed=61, **kw)
        dd = D.DeviceDrafter(SHAPE, w)
        # float64 copies of the head's operands, so the oracle's per-step products do not convert
        # the 151936-row matrices again at every step (np.asarray of a float64 array is a no-op)
        w64 = {k: np.asarray(w[k], np.float64) for k in ("embed", "ar_E", "ar_W")}
        _CACHE[regime] = (w, dd, w64)
    return _CACHE[regime]


def _inputs(B, seed):
    g, H, V = SHAPE.gamma, SHAPE.hidden, SHAPE.vocab
    rng = np.random.default_rng(seed)
    reps = rng.standard_normal((B, g + 1, g, H)).astype(np.float32)
    acc = rng.integers(0, g + 1, B).astype(np.int32)
    bon = rng.integers(0, V, B).astype(np.int32)
    return reps, acc, bon


@pytest.mark.parametrize("B", [1, 2, 16, 20])
def test_full_head_at_qwen3_vocabulary(B):
    from paper_2609_27396_amd import dpara as D
    w, dd, w64 = _setup("full")
    g, H, V = SHAPE.gamma, SHAPE.hidden, SHAPE.vocab
    path = "single-launch head" if B <= 16 else "step kernels"
    _say(f"case full head, vocab {V}, gamma {g}, batch {B} ({path})")
    reps_h, acc_h, bon_h = _inputs(B, seed=100 + B)
    reps = torch.from_numpy(reps_h).cuda()
    acc, bon = torch.from_numpy(acc_h).cuda(), torch.from_numpy(bon_h).cuda()
    ws = D.Workspace(dd.cfg, B, 64)
    i32 = dict(dtype=torch.int32, device="cuda")
    gathered = torch.empty((B, g, H), dtype=torch.float32, device="cuda")
    drafts, nsp = torch.empty((B, g), **i32), torch.empty((B, g + 1), **i32)
    margins = torch.empty((B, g), dtype=torch.float32, device="cuda")
    scores = torch.empty((B, g, V), dtype=torch.float32, device="cuda")

    D.select_and_head(dd, reps, acc, bon, gathered, drafts, nsp, margins, ws)
    torch.cuda.synchronize()
    assert ws.status() == 0, ws.status()          # no timeout of the single-launch head either
    assert ws.head_fallback() != 0                 # the bound failed: the full head ran
    gh = gathered.cpu().numpy()
    for b in range(B):
        np.testing.assert_array_equal(gh[b], reps_h[b, acc_h[b]])  # bit-exact gather
    greedy = (drafts.cpu().numpy(), nsp.cpu().numpy(), margins.cpu().numpy())
    assert np.array_equal(greedy[1][:, 0], bon_h) and np.array_equal(greedy[1][:, 1:], greedy[0])

    T, seed = 0.9, 4242
    scores.fill_(float("nan"))
    D.select_and_head_sampled(dd, reps, acc, bon, None, drafts, nsp, None, T, seed, scores, ws)
    torch.cuda.synchronize()
    assert ws.status() == 0, ws.status()
    assert ws.head_fallback() != 0
    sampled = (drafts.cpu().numpy(), nsp.cpu().numpy())
    assert np.array_equal(sampled[1][:, 1:], sampled[0])

    # one product for every gathered row of the batch: l = h embed^T (the oracle's base logits)
    ell = O.base_logits(w64, gh.reshape(B * g, H), "bf16").reshape(B, g, V)
    comp, skip, comp_s, skip_s = 0, 0, 0, 0
    for b in range(B):
        y_prev = ys_prev = int(bon_h[b])
        sg = scores[b].cpu().numpy()
        for i in range(1, g + 1):
            y, m, _ = O.head_step(w64, ell[b, i - 1], y_prev, "bf16")
            if m > MARGIN:
                assert int(greedy[0][b, i - 1]) == y, (b, i, greedy[0][b, i - 1], y, m)
                assert abs(float(greedy[2][b, i - 1]) - m) < 1e-3 + 1e-3 * abs(m)
                comp += 1
            else:
                skip += 1
            y_prev = int(greedy[0][b, i - 1])
            ys, ms, s = O.head_step_sampled(w64, ell[b, i - 1], ys_prev, T, seed, b, i, "bf16")
            assert np.all(np.abs(sg[i - 1] - s) <= 1e-3 + 1e-3 * np.abs(s)), (b, i)
            if ms > MARGIN:
                assert int(sampled[0][b, i - 1]) == ys, (b, i, sampled[0][b, i - 1], ys, ms)
                comp_s += 1
            else:
                skip_s += 1
            ys_prev = int(sampled[0][b, i - 1])
    _say(f"batch {B}: greedy steps compared {comp} (skipped {skip}), sampled {comp_s} (skipped {skip_s})")
    assert skip <= max(1, B * g // 20) and skip_s <= max(1, B * g // 20)
    assert not np.array_equal(sampled[0], greedy[0])  # the noise reaches the draws

    if B == 16:
        # the off-serial-path variant hands over to the same full head: the same bits
        cand = D.branch_candidates_buffer(dd, B)
        D.branch_candidates(dd, reps, cand, ws)
        d2, n2 = torch.empty_like(drafts), torch.empty_like(nsp)
        m2, g2 = torch.empty_like(margins), torch.empty_like(gathered)
        D.select_and_head_cand(dd, reps, cand, acc, bon, g2, d2, n2, m2, ws)
        torch.cuda.synchronize()
        assert ws.status() == 0 and ws.head_fallback() != 0
        assert np.array_equal(d2.cpu().numpy(), greedy[0]) and np.array_equal(n2.cpu().numpy(), greedy[1])
        assert np.array_equal(m2.cpu().numpy(), greedy[2]) and np.array_equal(g2.cpu().numpy(), gh)
    if B * g > 128:
        # with the embedding's max row norm prepared, the plain greedy head over more than 128
        # gathered rows ranks by the hi parts first; here no step is proven, so it hands over to
        # the same LM head and full head: the same bits
        dd.prepare_candidates(ws)
        d3, n3 = torch.empty_like(drafts), torch.empty_like(nsp)
        m3, g3 = torch.empty_like(margins), torch.empty_like(gathered)
        D.select_and_head(dd, reps, acc, bon, g3, d3, n3, m3, ws)
        torch.cuda.synchronize()
        dd.unprepare_candidates()
        assert ws.status() == 0 and ws.head_fallback() != 0
        assert np.array_equal(d3.cpu().numpy(), greedy[0]) and np.array_equal(n3.cpu().numpy(), greedy[1])
        assert np.array_equal(m3.cpu().numpy(), greedy[2]) and np.array_equal(g3.cpu().numpy(), gh)


@pytest.mark.parametrize("B", [1, 2, 4, 9, 13, 16])
def test_candidates_head_at_qwen3_vocabulary(B):
    """The off-serial-path head at the Qwen3 vocabulary with the default weight scales: every
    branch row ranked by its bf16 hi part, the 16 candidates rescored with hi + lo, the bound
    widened by the lo part's and the rounding's share.  Where neither head falls back, the
    drafts, margins and next spine are bit for bit those of the plain head (whose candidates
    come from the two-plane LM head), so the rescored logits are the LM head's; the prepared
    max |embed_v|^2 gives the same bits as the per-call pass; and the drafts agree with the
    oracle wherever its top1 - top2 margin exceeds 1e-2."""
    from paper_2609_27396_amd import dpara as D
    w, dd, w64 = _setup("pruned")
    g, H, V = SHAPE.gamma, SHAPE.hidden, SHAPE.vocab
    _say(f"case candidates head, vocab {V}, gamma {g}, batch {B}")
    reps_h, acc_h, bon_h = _inputs(B, seed=300 + B)
    reps = torch.from_numpy(reps_h).cuda()
    acc, bon = torch.from_numpy(acc_h).cuda(), torch.from_numpy(bon_h).cuda()
    ws = D.Workspace(dd.cfg, B, 64)
    i32 = dict(dtype=torch.int32, device="cuda")

    def outs():
        return (torch.empty((B, g), **i32), torch.empty((B, g + 1), **i32),
                torch.empty((B, g), dtype=torch.float32, device="cuda"),
                torch.empty((B, g, H), dtype=torch.float32, device="cuda"))

    d0, n0, m0, g0 = outs()
    D.select_and_head(dd, reps, acc, bon, g0, d0, n0, m0, ws)
    torch.cuda.synchronize()
    fb_plain = ws.head_fallback()
    runs = []
    for prepared in (False, True):
        if prepared:
            dd.prepare_candidates(ws)
            torch.cuda.synchronize()
            e2 = float(dd.enorm2.item())
            ref = float((w["embed"].astype(np.float64) ** 2).sum(1).max())
            assert abs(e2 / ref - 1) < 1e-5, (e2, ref)
        cand = D.branch_candidates_buffer(dd, B)
        D.branch_candidates(dd, reps, cand, ws)
        d1, n1, m1, g1 = outs()
        D.select_and_head_cand(dd, reps, cand, acc, bon, g1, d1, n1, m1, ws)
        torch.cuda.synchronize()
        assert ws.status() == 0
        runs.append((ws.head_fallback(), d1.cpu(), n1.cpu(), m1.cpu(), g1.cpu()))
    # the plain head again, now with the norm prepared: above 128 gathered rows it ranks by the
    # hi parts and rescores (the same machinery over the accepted rows only)
    d4, n4, m4, g4 = outs()
    D.select_and_head(dd, reps, acc, bon, g4, d4, n4, m4, ws)
    torch.cuda.synchronize()
    fb_ranked = ws.head_fallback()
    dd.unprepare_candidates()
    assert torch.equal(g4.cpu(), g0.cpu())
    if fb_ranked == 0 and fb_plain == 0:
        for a, b in zip((d4.cpu(), n4.cpu(), m4.cpu()), (d0.cpu(), n0.cpu(), m0.cpu())):
            assert torch.equal(a, b)
    fb = runs[0][0]
    _say(f"batch {B}: fallback flags plain {fb_plain}, candidates {fb}")
    for a, b in zip(runs[0], runs[1]):
        assert torch.equal(a, b) if isinstance(a, torch.Tensor) else a == b
    assert torch.equal(runs[0][4], g0.cpu())
    if fb == 0 and fb_plain == 0:
        for a, b in zip(runs[0][1:4], (d0.cpu(), n0.cpu(), m0.cpu())):
            assert torch.equal(a, b)
    if B == 1:
        assert fb == 0  # one request: every step proven under the widened bound
    drafts, margins = runs[0][1].numpy(), runs[0][3].numpy()
    gh = runs[0][4].numpy()
    ell = O.base_logits(w64, gh.reshape(B * g, H), "bf16").reshape(B, g, V)
    comp = skip = 0
    for b in range(B):
        y_prev = int(bon_h[b])
        for i in range(1, g + 1):
            y, m, _ = O.head_step(w64, ell[b, i - 1], y_prev, "bf16")
            if m > MARGIN:
                assert int(drafts[b, i - 1]) == y, (b, i, drafts[b, i - 1], y, m)
                assert abs(float(margins[b, i - 1]) - m) < 1e-3 + 1e-3 * abs(m)
                comp += 1
            else:
                skip += 1
            y_prev = int(drafts[b, i - 1])
    _say(f"batch {B}: steps compared {comp} (skipped {skip})")
    assert skip <= max(1, B * g // 10)  # (near ties are more frequent at these small AR scales)
