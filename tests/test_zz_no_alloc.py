"""dpara_verify_greedy_noalloc (the verification for callers that cannot allocate: its scratch is
the library's static device array) against dpara_verify_greedy (workspace scratch), through the
C ABI: two calls in a row, the second with a smaller input, every output bit for bit; the
verdicts also equal the planted ones and the oracle's."""
import types

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import dpara_oracle as O  # noqa: E402
from paper_2609_27396_amd import synth  # noqa: E402

pytestmark = pytest.mark.gpu


def _one_call(B, V, gamma, logits_dtype, seed):
    from paper_2609_27396_amd import dpara as D
    shape = synth.DrafterShape(n_layers=1, hidden=256, n_q_heads=2, n_kv_heads=1, head_dim=128, ffn=512,
                               vocab=V, gamma=gamma, ar_rank=64, qk_norm=True, dtype="bf16")
    wl = synth.Workload("na", shape, batch=B, ctx_min=0, ctx_max=0, p_reject=0.2, seed_in=seed,
                        logits_dtype=logits_dtype)
    rng = synth._rng(seed, 7)
    spine = rng.integers(0, V, size=(B, gamma + 1)).astype(np.int32)
    acc_p = synth.accepted_lengths(rng, B, gamma, wl.p_reject)
    T, bonus_p = synth.plant_target_logits(rng, spine, acc_p, V, logits_dtype == "bf16")
    d = types.SimpleNamespace(cfg=D.make_config(shape))
    tl = torch.from_numpy(T).cuda().to(torch.bfloat16 if logits_dtype == "bf16" else torch.float32)
    sp = torch.from_numpy(spine).cuda()
    i32 = dict(dtype=torch.int32, device="cuda")
    out_ws = [torch.full((B,), -7, **i32), torch.full((B,), -7, **i32), torch.full((B, gamma + 1), -7, **i32)]
    out_na = [torch.full((B,), -9, **i32), torch.full((B,), -9, **i32), torch.full((B, gamma + 1), -9, **i32)]
    ws = D.Workspace(d.cfg, B, 64)
    D.verify_greedy(d, tl, sp, *out_ws, ws)
    status = torch.zeros(1, **i32)
    D.verify_greedy_noalloc(d, tl, sp, *out_na, status=status)
    torch.cuda.synchronize()
    assert ws.status() == 0 and int(status.item()) == 0
    for a, b in zip(out_ws, out_na):
        assert torch.equal(a, b)
    acc, bon = out_na[0].cpu().numpy(), out_na[1].cpu().numpy()
    assert np.array_equal(acc, acc_p) and np.array_equal(bon, bonus_p)
    for b in range(B):
        r, bonus, g = O.verify_greedy(T[b], spine[b])
        assert (int(acc[b]), int(bon[b])) == (r, bonus)
        np.testing.assert_array_equal(out_na[2][b].cpu().numpy(), g)
    return d, tl, sp, out_na


def test_noalloc_verify_matches_workspace_verify():
    # first call: Qwen3 vocabulary, 12 requests, bf16 logits (partials in most of the scratch's head)
    _one_call(12, 151936, 16, "bf16", seed=3)
    # second call, smaller: 3 requests, vocabulary 5000, float32 logits; the scratch keeps the
    # first call's partials beyond what this call writes, which it must never read
    d, tl, sp, out = _one_call(3, 5000, 7, "f32", seed=4)
    # status: an out-of-range draft sets the range bit in the caller's word (and never matches);
    # without a status pointer the call still runs and gives the same outputs
    from paper_2609_27396_amd import dpara as D
    bad = sp.clone()
    bad[1, 1] = 5000 + 11
    i32 = dict(dtype=torch.int32, device="cuda")
    status = torch.zeros(1, **i32)
    a1, b1 = torch.empty(3, **i32), torch.empty(3, **i32)
    D.verify_greedy_noalloc(d, tl, bad, a1, b1, status=status)
    a2, b2 = torch.empty(3, **i32), torch.empty(3, **i32)
    D.verify_greedy_noalloc(d, tl, bad, a2, b2)
    torch.cuda.synchronize()
    assert int(status.item()) & D.STATUS_TOKEN_RANGE
    assert int(a1[1]) == 0 and torch.equal(a1, a2) and torch.equal(b1, b2)
    assert torch.equal(a1[0::2], out[0][0::2])
