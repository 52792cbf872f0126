"""GPU parity of the sampling variant (speculative-sampling verification and the sampled AR
head) against the oracle, through the C ABI.

Both sides draw from the same counter-based generator, so the draws are the same wherever
floating point cannot flip them: an acceptance test is compared where the oracle's log-ratio
margin |log p - log q - log u| exceeds 1e-4 (the float32 log-sum-exp over the vocabulary is
good to about 1e-6 there), a bonus or head draw where the oracle's top1 - top2 of the
perturbed scores exceeds 1e-3 (bonus) or 1e-2 (head, whose scores carry the bf16 model's
rounding); the tests also require that almost every decision was compared."""
import types

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import dpara_oracle as O  # noqa: E402
from paper_2609_27396_amd import synth  # noqa: E402

pytestmark = pytest.mark.gpu

ACC_MARGIN, BONUS_MARGIN, HEAD_MARGIN = 1e-4, 1e-3, 1e-2


def _say(*a):
    print(*a, flush=True)


def _round_bf16(x):
    return torch.from_numpy(np.asarray(x, np.float32)).to(torch.bfloat16).float().numpy()


def _verify_inputs(B, gamma, V, T, dtype, seed):
    """Target logits N(0, 2); draft scores close to the target's tempered logits for even
    requests (long acceptances) and unrelated for odd ones; drafts drawn from q."""
    rng = np.random.default_rng(seed)
    L = rng.standard_normal((B, gamma + 1, V)).astype(np.float32) * 2.0
    if dtype == "bf16":
        L = _round_bf16(L)
    S = np.empty((B, gamma, V), np.float32)
    for b in range(B):
        if b % 2 == 0:
            S[b] = L[b, :gamma] / T + rng.standard_normal((gamma, V)).astype(np.float32) * 0.3
        else:
            S[b] = rng.standard_normal((gamma, V)).astype(np.float32) * 2.0
    spine = np.empty((B, gamma + 1), np.int32)
    spine[:, 0] = rng.integers(0, V, B)
    for b in range(B):
        for i in range(gamma):
            q = np.exp(S[b, i].astype(np.float64) - S[b, i].max())
            spine[b, i + 1] = rng.choice(V, p=q / q.sum())
    return L, S, spine


VERIFY_CASES = {
    "v3001_bf16_t1": (6, 5, 3001, 1.0, "bf16"),     # odd vocabulary: element loads
    "v8192_f32_t07": (5, 7, 8192, 0.7, "f32"),      # 16-byte loads, temperature 0.7
    "v151936_bf16_t1": (2, 16, 151936, 1.0, "bf16"),  # Qwen3 vocabulary, draft length 16
    "v1000_bf16_g63": (3, 63, 1000, 1.0, "bf16"),   # the longest draft the library takes
}


@pytest.mark.parametrize("case", sorted(VERIFY_CASES))
def test_verify_sampled_parity(case):
    from paper_2609_27396_amd import dpara as D
    B, gamma, V, T, dtype = VERIFY_CASES[case]
    shape = synth.DrafterShape(n_layers=1, hidden=256, n_q_heads=2, n_kv_heads=1, head_dim=128, ffn=512,
                               vocab=V, gamma=gamma, ar_rank=64, qk_norm=True, dtype="bf16")
    _say("case", case)
    cfg = D.make_config(shape)
    d = types.SimpleNamespace(cfg=cfg)
    ws = D.Workspace(cfg, B, 64)
    L, S, spine = _verify_inputs(B, gamma, V, T, dtype, seed=len(case))
    tl = torch.from_numpy(L).cuda().to(torch.bfloat16 if dtype == "bf16" else torch.float32)
    sc = torch.from_numpy(S).cuda()
    sp = torch.from_numpy(spine).cuda()
    acc = torch.empty(B, dtype=torch.int32, device="cuda")
    bon = torch.empty(B, dtype=torch.int32, device="cuda")
    compared, total, accepted = 0, 0, []
    for seed in (1, 2, 0xDEADBEEF12345):
        D.dpara_clear_status(ws.ptr, D._stream(None))
        D.verify_sampled(d, tl, sc, sp, T, seed, acc, bon, ws)
        torch.cuda.synchronize()
        assert ws.status() == 0
        ga, gb = acc.cpu().numpy(), bon.cpu().numpy()
        for b in range(B):
            r, bonus, info = O.verify_sampled(L[b], S[b], spine[b], T, seed, b)
            am = np.abs(info["accept_margins"])
            total += 1
            accepted.append(int(ga[b]))
            if am.min() > ACC_MARGIN:
                assert int(ga[b]) == r, (seed, b, ga[b], r, info["accept_margins"])
                if info["bonus_margin"] > BONUS_MARGIN:
                    assert int(gb[b]) == bonus, (seed, b, gb[b], bonus, info["bonus_margin"])
                    compared += 1
    _say(f"{case}: accepted lengths {accepted}; compared {compared} of {total} verdicts")
    assert compared >= total - 1
    assert max(accepted) >= 2 and min(accepted) == 0


def test_verify_sampled_full_acceptance_and_token_range():
    """q == p accepts every draft and draws the bonus from p_gamma; an out-of-range draft is
    flagged and never accepted."""
    from paper_2609_27396_amd import dpara as D
    B, gamma, V, T = 3, 4, 1000, 1.0
    shape = synth.DrafterShape(n_layers=1, hidden=256, n_q_heads=2, n_kv_heads=1, head_dim=128, ffn=512,
                               vocab=V, gamma=gamma, ar_rank=64, qk_norm=True, dtype="bf16")
    cfg = D.make_config(shape)
    d = types.SimpleNamespace(cfg=cfg)
    ws = D.Workspace(cfg, B, 64)
    L = np.random.default_rng(3).standard_normal((B, gamma + 1, V)).astype(np.float32)
    S = np.ascontiguousarray(L[:, :gamma])
    spine = np.random.default_rng(4).integers(0, V, (B, gamma + 1)).astype(np.int32)
    acc = torch.empty(B, dtype=torch.int32, device="cuda")
    bon = torch.empty(B, dtype=torch.int32, device="cuda")
    D.verify_sampled(d, torch.from_numpy(L).cuda(), torch.from_numpy(S).cuda(), torch.from_numpy(spine).cuda(), T,
                     9, acc, bon, ws)
    torch.cuda.synchronize()
    assert ws.status() == 0
    for b in range(B):
        r, bonus, info = O.verify_sampled(L[b], S[b], spine[b], T, 9, b)
        assert r == gamma and int(acc[b]) == gamma
        if info["bonus_margin"] > BONUS_MARGIN:
            assert int(bon[b]) == bonus
    spine[1, 2] = V + 7
    D.verify_sampled(d, torch.from_numpy(L).cuda(), torch.from_numpy(S).cuda(), torch.from_numpy(spine).cuda(), T,
                     9, acc, bon, ws)
    torch.cuda.synchronize()
    assert ws.status() & D.STATUS_TOKEN_RANGE
    assert int(acc[1]) == 1 and int(acc[0]) == gamma


def _check_head_sampled(shape, w, dr, scores, T, seed, mode):
    """Teacher-forced: step i of the oracle is fed the GPU's y_{i-1} and the GPU's gathered
    rows (copied bit for bit from its reps); scores within 1e-3 + 1e-3 |s|."""
    compared = 0
    for b in range(dr.B):
        gathered = dr.gathered[b].cpu().numpy()
        r = int(dr.accept[b].item())
        np.testing.assert_array_equal(gathered, dr.reps[b, r].cpu().numpy())
        drafts, bonus = dr.drafts[b].cpu().numpy(), int(dr.bonus[b].item())
        assert dr.next_spine[b, 0].item() == bonus
        np.testing.assert_array_equal(dr.next_spine[b, 1:].cpu().numpy(), drafts)
        sg = scores[b].cpu().numpy()
        ell = O.base_logits(w, gathered, mode)
        y_prev = bonus
        for i in range(1, shape.gamma + 1):
            y, m, s = O.head_step_sampled(w, ell[i - 1], y_prev, T, seed, b, i, mode)
            assert np.all(np.abs(sg[i - 1] - s) <= 1e-3 + 1e-3 * np.abs(s)), (b, i)
            if m > HEAD_MARGIN:
                assert int(drafts[i - 1]) == y, (b, i, drafts[i - 1], y, m)
                compared += 1
            y_prev = int(drafts[i - 1])
    return compared


HEAD_CASES = {
    # (shape, contexts, temperature, std of the head's W).  A large W defeats the pruned steps'
    # bound, so the full sampled head runs: bf16, rank 64, 3 requests: the single-launch head
    "bf16_persistent": ("h256_hd128_g5", [0, 77, 300], 1.0, 0.3),
    # bf16, 18 requests (more than one persistent launch holds): the step kernels
    "bf16_steps_b18": ("h256_hd128_g5", [5 * i for i in range(18)], 0.8, 0.3),
    # float32 model: the step kernels
    "f32_steps": ("f32_h256_g7", [33, 150], 1.0, 0.3),
    # a small W: every step is proven over the perturbed logits' candidates, and the scores
    # come from the scores kernel
    "bf16_pruned": ("h256_hd128_g5", [0, 77, 300], 1.0, 0.005),
    "f32_pruned": ("f32_h256_g7", [33, 150], 0.7, 0.005),
}


@pytest.mark.parametrize("case", sorted(HEAD_CASES))
def test_head_sampled_parity(case):
    from test_gpu_parity import SMALL_CASES
    from paper_2609_27396_amd.harness import DeviceRound
    name, ctx, T, w_std = HEAD_CASES[case]
    shape = SMALL_CASES[name][0]
    mode = shape.dtype
    _say("case", case)
    wl = synth.Workload("hs", shape, batch=len(ctx), ctx_min=0, ctx_max=0, p_reject=0.3, seed_in=21,
                        logits_dtype="bf16" if mode == "bf16" else "f32")
    w = synth.make_weights(shape, seed=22, gain_jitter=0.1, ar_e_std=1.0, ar_w_std=w_std)
    ri = synth.make_round(wl, ctx_lens=ctx)
    dr = DeviceRound(shape, w, ri)
    dr.backbone()
    dr.verify()
    scores = torch.empty((len(ctx), shape.gamma, shape.vocab), dtype=torch.float32, device="cuda")
    total = 0
    for seed in (5, 77):
        scores.fill_(float("nan"))
        dr.head_sampled(T, seed, scores)
        torch.cuda.synchronize()
        assert dr.status() == 0
        assert (dr.head_fallback() != 0) == (w_std > 0.1), dr.head_fallback()  # which path ran
        compared = _check_head_sampled(shape, w, dr, scores, T, seed, mode)
        total += len(ctx) * shape.gamma
        _say(f"{case} seed {seed}: drafts {dr.drafts.cpu().numpy().tolist()[:3]}, compared {compared}")
        assert compared >= len(ctx) * shape.gamma - 2
    # the draws are not the greedy tokens (the noise is there) and differ between seeds
    dr.head_sampled(T, 5, scores)
    d5 = dr.drafts.clone()
    dr.head_sampled(T, 6, scores)
    assert not torch.equal(d5, dr.drafts)
    # scores may be NULL
    dr.head_sampled(T, 5, None)
    torch.cuda.synchronize()
    assert torch.equal(d5, dr.drafts)


def test_iterated_sampled_rounds():
    """Algorithm 1 with sampling, iterated over three rounds on random weights: target forward
    of the block (hidden states after layers 0, 1 and 3), speculative-sampling verification
    against the draft scores the previous round's sampled head wrote, the all-boundary
    backbone, the sampled head (next block and its scores), fusion and the append of
    t_0..t_r.  The loop is driven by the oracle's own decisions (block, append count); the
    GPU's verdict, bonus and drafts are compared with the oracle's wherever its margins make
    them unique, its scores within the head's bar.  Round 0 starts from synthetic scores."""
    from test_gpu_parity import LOOP_DRAFTER, LOOP_TARGET, FEAT_LAYERS, TOL
    from paper_2609_27396_amd import dpara as D
    from paper_2609_27396_amd.harness import DeviceRound, upload_cache
    sd, st_ = LOOP_DRAFTER, LOOP_TARGET
    ctx_lens, B, g, H, V, T = [40, 75], 2, sd.gamma, sd.hidden, sd.vocab, 1.0
    nf = len(FEAT_LAYERS)
    wd = synth.make_weights(sd, seed=41, gain_jitter=0.1, ar_e_std=1.0, ar_w_std=0.3)
    wt = synth.make_target_weights(st_, seed=42, gain_jitter=0.1)
    wf = synth.make_fusion_weights(sd, n_feat=nf, seed=43, gain_jitter=0.1)
    wl = synth.Workload("sloop", sd, batch=B, ctx_min=0, ctx_max=0, p_reject=0.3, seed_in=44)
    ri = synth.make_round(wl, ctx_lens=ctx_lens)
    dr = DeviceRound(sd, wd, ri, ctx_cap=256)
    tk, tv = synth.make_target_cache(st_, ctx_lens, seed=45)
    t = D.DeviceTarget(st_, wt)
    tctx = D.DeviceContext(st_, B, 256)
    upload_cache(tctx, tk, tv, ctx_lens, torch.bfloat16)
    tws = D.Workspace(t.cfg, B, 256, target=True)
    fus = D.DeviceFusion(sd, wf, nf)
    fws = torch.empty(D.dpara_fuse_workspace_bytes(fus.cfg, B * (g + 1), nf), dtype=torch.uint8, device="cuda")
    hid = torch.empty((B, g + 1, nf, H), dtype=torch.bfloat16, device="cuda")
    fused = torch.empty((B, g + 1, H), dtype=torch.bfloat16, device="cuda")
    scores_in = torch.empty((B, g, V), dtype=torch.float32, device="cuda")
    scores_out = torch.empty_like(scores_in)
    feats = [np.asarray(f, np.float32) for f in ri.ctx_feats]
    spine = ri.spine.astype(np.int32).copy()
    s_ref = np.random.default_rng(46).standard_normal((B, g, V)).astype(np.float32)  # round 0's q
    scores_in.copy_(torch.from_numpy(s_ref))
    stats = {"verdicts": 0, "bonus": 0, "drafts": 0, "accepted": []}
    for rnd in range(3):
        seed = 1000 + rnd
        dr.spine.copy_(torch.from_numpy(spine))
        D.target_forward_hidden(t, tctx, dr.spine, dr.logits, FEAT_LAYERS, hid, tws)
        dr.verify_sampled(scores_in, T, seed)
        dr.backbone()
        dr.head_sampled(T, seed, scores_out)
        D.fuse_features(fus, hid.view(B * (g + 1), nf * H), fused.view(B * (g + 1), H), fws)
        torch.cuda.synchronize()
        assert dr.status() == 0
        acc, bon, drafts = dr.accept.cpu().numpy(), dr.bonus.cpu().numpy(), dr.drafts.cpu().numpy()
        sc_gpu = scores_out.cpu().numpy()
        nxt, n_new, s_next = np.zeros_like(spine), np.zeros(B, np.int32), np.zeros((B, g, V), np.float32)
        for b in range(B):
            tl, th = O.target_forward(st_, wt, [tk[l][b] for l in range(st_.n_layers)],
                                      [tv[l][b] for l in range(st_.n_layers)], spine[b], "bf16", FEAT_LAYERS)
            r, bonus, info = O.verify_sampled(tl, s_ref[b], spine[b], T, seed, b)
            if np.abs(info["accept_margins"]).min() > 2e-2:   # the GPU's logits and scores carry bf16 error
                assert int(acc[b]) == r, (rnd, b, acc[b], r)
                stats["verdicts"] += 1
                if info["bonus_margin"] > 5e-2:
                    assert int(bon[b]) == bonus, (rnd, b)
                    stats["bonus"] += 1
            stats["accepted"].append(int(acc[b]))
            ref = O.backbone_all_boundaries(sd, wd, feats[b], spine[b], "bf16")["reps"]
            hd = O.select_and_head_sampled(sd, wd, ref, r, bonus, T, seed, b, "bf16")
            if (int(acc[b]), int(bon[b])) == (r, bonus):
                for i in range(g):               # the oracle's own chain, up to its first near-tie
                    if hd["margins"][i] <= 5e-2:
                        break
                    assert int(drafts[b, i]) == int(hd["drafts"][i]), (rnd, b, i)
                    stats["drafts"] += 1
                    # the score row the draw came from
                    assert np.all(np.abs(sc_gpu[b, i] - hd["scores"][i]) <= 2e-2 + 2e-2 * np.abs(hd["scores"][i]))
            k = r + 1
            f_ref = O.fuse_features(sd, wf, th[:k].reshape(k, nf * H), "bf16")
            feats[b] = np.concatenate([feats[b], f_ref.astype(np.float32)])
            nxt[b], n_new[b], s_next[b] = hd["next_spine"], k, hd["scores"]
        nn = torch.from_numpy(n_new).cuda()
        dr.append(nn, fused)
        # the next round's verification reads the scores of the block it verifies: the GPU's
        # own when its block is the GPU's, else the oracle's (the loop follows the oracle)
        same = [bool(np.array_equal(nxt[b], dr.next_spine[b].cpu().numpy())) for b in range(B)]
        for b in range(B):
            if not same[b]:
                scores_out[b].copy_(torch.from_numpy(s_next[b]))
        scores_in.copy_(scores_out)
        s_ref, spine = s_next, nxt
        _say(f"sampled round {rnd}: accepted {acc.tolist()} (oracle-driven), same next block {same}")
    _say("iterated sampled rounds:", stats)
    assert stats["verdicts"] >= 4 and stats["drafts"] >= 4


def _freq_ok(counts, p, sig=5.0):
    n = counts.sum()
    f = counts / n
    return np.all(np.abs(f - p) <= sig * np.sqrt(p * (1 - p) / n) + 1.0 / n)


def test_verify_sampled_preserves_target_distribution():
    """The GPU's own draws, as a distribution: 4096 requests share one target and draft
    distribution (each request index is its own random stream), drafts drawn from q; the first
    and second emitted tokens follow p_0 and p_1 and t_1 is accepted at rate sum min(p, q)."""
    from paper_2609_27396_amd import dpara as D
    B, gamma, V, T = 4096, 2, 8, 1.0
    shape = synth.DrafterShape(n_layers=1, hidden=256, n_q_heads=2, n_kv_heads=1, head_dim=128, ffn=512,
                               vocab=V, gamma=gamma, ar_rank=64, qk_norm=True, dtype="bf16")
    cfg = D.make_config(shape)
    d = types.SimpleNamespace(cfg=cfg)
    ws = D.Workspace(cfg, B, 64)
    rng = np.random.default_rng(17)
    L1 = rng.standard_normal((gamma + 1, V)).astype(np.float32) * 1.5
    S1 = rng.standard_normal((gamma, V)).astype(np.float32) * 1.5
    p = [np.exp(L1[j] - L1[j].max()) / np.exp(L1[j] - L1[j].max()).sum() for j in range(gamma + 1)]
    q = [np.exp(S1[j] - S1[j].max()) / np.exp(S1[j] - S1[j].max()).sum() for j in range(gamma)]
    spine = np.zeros((B, gamma + 1), np.int32)
    for i in range(gamma):
        spine[:, i + 1] = rng.choice(V, size=B, p=q[i])
    L = np.ascontiguousarray(np.broadcast_to(L1, (B, gamma + 1, V)))
    S = np.ascontiguousarray(np.broadcast_to(S1, (B, gamma, V)))
    acc = torch.empty(B, dtype=torch.int32, device="cuda")
    bon = torch.empty(B, dtype=torch.int32, device="cuda")
    D.verify_sampled(d, torch.from_numpy(L).cuda(), torch.from_numpy(S).cuda(), torch.from_numpy(spine).cuda(), T,
                     31337, acc, bon, ws)
    torch.cuda.synchronize()
    assert ws.status() == 0
    r, b = acc.cpu().numpy(), bon.cpu().numpy()
    e1 = np.where(r >= 1, spine[:, 1], b)
    e2 = np.where(r >= 2, spine[:, 2], b)[r >= 1]
    assert _freq_ok(np.bincount(e1, minlength=V), p[0])
    assert _freq_ok(np.bincount(e2, minlength=V), p[1])
    a = float(np.minimum(p[0], q[0]).sum())
    assert abs((r >= 1).mean() - a) <= 5 * np.sqrt(a * (1 - a) / B)
    _say(f"acceptance of t_1 {(r >= 1).mean():.4f} (sum min(p, q) = {a:.4f}); mean accepted {r.mean():.3f}")


@pytest.mark.parametrize("batch", [16, 512])
def test_head_sampled_draws_follow_softmax(batch):
    """With the head's correction matrix W zero, each sampled step is a plain draw from
    softmax(l_i / T): over many requests (16: the single-launch head; 512: the step kernels)
    the draws of every step follow it."""
    from paper_2609_27396_amd import dpara as D
    shape = synth.DrafterShape(n_layers=1, hidden=256, n_q_heads=2, n_kv_heads=1, head_dim=128, ffn=512,
                               vocab=64, gamma=3, ar_rank=64, qk_norm=True, dtype="bf16")
    w = synth.make_weights(shape, seed=8, weight_std=0.1)
    w["ar_W"] = np.zeros_like(w["ar_W"])
    dd = D.DeviceDrafter(shape, w)
    B, g, H, V, T = batch, shape.gamma, shape.hidden, shape.vocab, 0.8
    ws = D.Workspace(dd.cfg, B, 64)
    rows = np.random.default_rng(9).standard_normal((g, H)).astype(np.float32)
    reps = torch.from_numpy(np.ascontiguousarray(np.broadcast_to(rows, (B, g + 1, g, H)))).cuda()
    acc = torch.zeros(B, dtype=torch.int32, device="cuda")
    bon = torch.zeros(B, dtype=torch.int32, device="cuda")
    drafts = torch.empty((B, g), dtype=torch.int32, device="cuda")
    nsp = torch.empty((B, g + 1), dtype=torch.int32, device="cuda")
    counts = np.zeros((g, V))
    for seed in range(4096 // B if B < 4096 else 1):
        D.select_and_head_sampled(dd, reps, acc, bon, None, drafts, nsp, None, T, seed, None, ws)
        dh = drafts.cpu().numpy()
        for i in range(g):
            counts[i] += np.bincount(dh[:, i], minlength=V)
    torch.cuda.synchronize()
    assert ws.status() == 0
    ell = O.base_logits(w, rows, "bf16") / T
    for i in range(g):
        pz = np.exp(ell[i] - ell[i].max())
        assert _freq_ok(counts[i], pz / pz.sum()), i
