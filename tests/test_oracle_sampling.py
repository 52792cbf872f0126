"""Pins of the oracle's sampling variant (no GPU needed): the counter-based generator
against its published known answers, the uniform and Gumbel transforms against their
distributions, the sampled head against its greedy and noise-free special cases, and the
speculative-sampling verification against the property that defines it (the emitted tokens
follow the target's distributions, whatever the drafter's) plus the closed-form acceptance
rate sum_v min(p(v), q(v)).  Monte Carlo bounds are 5 standard deviations."""
import os

import numpy as np

from oracle import dpara_oracle as O
from paper_2609_27396_amd import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _softmax(x):
    e = np.exp(np.asarray(x, np.float64) - np.max(x))
    return e / e.sum()


def _within(freq, p, n, sig=5.0):
    return np.all(np.abs(freq - p) <= sig * np.sqrt(p * (1 - p) / n) + 1.0 / n)


def test_philox_known_answers():
    rows = [l.split() for l in open(os.path.join(GOLDEN, "philox4x32_10_kat.txt")) if l.strip() and l[0] != "#"]
    assert len(rows) == 3
    for r in rows:
        x = [int(t, 16) for t in r]
        got = [int(w) for w in O.philox4x32_10(x[0:4], x[4:6])]
        assert got == x[6:10], r
    # vector form: counters broadcast along an array give the scalar results element by element
    ctr0 = np.array([0, 1, 2, 0xFFFFFFFF], np.uint64)
    vec = O.philox4x32_10((ctr0, 7, 8, 9), (11, 12))
    for k, c in enumerate(ctr0):
        assert [int(w[k]) for w in vec] == [int(w) for w in O.philox4x32_10((int(c), 7, 8, 9), (11, 12))]


def test_u01_range_and_moments():
    assert O.u01(0) == 2.0 ** -24 and O.u01(0xFFFFFFFF) == 1.0 - 2.0 ** -24
    assert float(np.float32(O.u01(0x12345678))) == O.u01(0x12345678)  # exact in float32
    n = 200_000
    u = O.uniforms(123, O.TAG_HEAD, 3, 5, np.arange(n))
    assert 0.0 < u.min() and u.max() < 1.0
    assert abs(u.mean() - 0.5) < 5 * np.sqrt(1 / 12 / n)
    assert abs(u.var() - 1 / 12) < 5 * np.sqrt((1 / 80 - 1 / 144) / n)  # sd of a sample variance
    hist = np.histogram(u, bins=16, range=(0, 1))[0]
    assert _within(hist / n, np.full(16, 1 / 16), n)
    # different tags, requests, positions and seeds give unrelated streams
    for other in (O.uniforms(123, O.TAG_BONUS, 3, 5, np.arange(n)), O.uniforms(123, O.TAG_HEAD, 4, 5, np.arange(n)),
                  O.uniforms(123, O.TAG_HEAD, 3, 6, np.arange(n)), O.uniforms(124, O.TAG_HEAD, 3, 5, np.arange(n))):
        assert abs(np.corrcoef(u, other)[0, 1]) < 5 / np.sqrt(n)


def test_gumbel_max_frequencies_follow_softmax():
    s = np.array([0.3, -1.2, 2.0, 0.0, 1.1, -0.4])
    n = 12_000
    counts = np.zeros(s.size)
    for i in range(n):
        counts[O.gumbel_argmax(s, 77, O.TAG_HEAD, 0, i)[0]] += 1
    assert _within(counts / n, _softmax(s), n)
    # -inf entries never win
    t = s.copy()
    t[2] = -np.inf
    assert all(O.gumbel_argmax(t, 5, O.TAG_BONUS, 1, i)[0] != 2 for i in range(300))


def test_sampled_head_special_cases():
    shape = synth.DrafterShape(n_layers=1, hidden=32, n_q_heads=2, n_kv_heads=1, head_dim=16, ffn=64, vocab=50,
                               gamma=3, ar_rank=8, qk_norm=True, dtype="f32")
    w = synth.make_weights(shape, seed=2, ar_e_std=1.0, ar_w_std=0.5)
    ell = np.random.default_rng(3).standard_normal(shape.vocab) * 2.0
    # without the correction term the step is a plain draw from softmax(l / T)
    w0 = dict(w, ar_W=np.zeros_like(w["ar_W"]))
    for i in range(1, 30):
        y, m, s = O.head_step_sampled(w0, ell, 7, 0.8, 99, 2, i, "exact")
        np.testing.assert_allclose(s, ell / 0.8, rtol=1e-15)
        assert (y, m) == O.gumbel_argmax(ell / 0.8, 99, O.TAG_HEAD, 2, i)
    # a temperature far below the top1 - top2 gap gives the greedy token
    for y_prev in range(20):
        yg, mg, _ = O.head_step(w, ell, y_prev, "exact")
        if mg > 0.2:
            assert O.head_step_sampled(w, ell, y_prev, 0.005, 1, 0, 1, "exact")[0] == yg
    # the draw changes with the step, request and seed, and the head feeds each draw forward
    reps = np.random.default_rng(4).standard_normal((shape.gamma + 1, shape.gamma, shape.hidden))
    hd = O.select_and_head_sampled(shape, w, reps, 1, 5, 1.0, 42, 0, "exact")
    ell1 = O.base_logits(w, reps[1], "exact")
    y_prev = 5
    for i in range(1, shape.gamma + 1):
        y, _, s = O.head_step_sampled(w, ell1[i - 1], y_prev, 1.0, 42, 0, i, "exact")
        assert hd["drafts"][i - 1] == y
        np.testing.assert_array_equal(hd["scores"][i - 1], s)
        y_prev = y
    assert list(hd["next_spine"]) == [5] + list(hd["drafts"])


def test_speculative_sampling_preserves_the_target():
    """Drafts drawn from q; the emitted tokens (accepted drafts, then the bonus) follow p at
    the first, second and third position, and t_1 is accepted with probability
    sum_v min(p_1(v), q_1(v))."""
    V, gam, T = 5, 2, 1.0
    rng = np.random.default_rng(8)
    L = np.array([[1.5, 0.2, -0.7, 0.0, 0.9], [-1.0, 0.3, 1.8, 0.4, -0.2], [0.1, 2.2, -0.5, -0.9, 0.6]])
    S = np.array([[0.2, 1.4, 0.0, -0.3, 0.5], [1.0, -0.8, 0.1, 1.6, 0.0]])
    p = [_softmax(L[j] / T) for j in range(gam + 1)]
    q = [_softmax(S[j]) for j in range(gam)]
    n = 8000
    e1, e2, e3, acc1 = np.zeros(V), np.zeros(V), np.zeros(V), 0
    for k in range(n):
        t1, t2 = rng.choice(V, p=q[0]), rng.choice(V, p=q[1])
        r, bonus, _ = O.verify_sampled(L, S, [0, t1, t2], T, 1234, k)
        emitted = [t1, t2][:r] + [bonus]
        e1[emitted[0]] += 1
        if r >= 1:
            acc1 += 1
            e2[emitted[1]] += 1
        if r == 2:
            e3[emitted[2]] += 1
    assert _within(e1 / n, p[0], n)
    assert _within(e2 / e2.sum(), p[1], int(e2.sum()))
    assert _within(e3 / e3.sum(), p[2], int(e3.sum()))
    a = float(np.minimum(p[0], q[0]).sum())
    assert abs(acc1 / n - a) <= 5 * np.sqrt(a * (1 - a) / n)


def test_verify_sampled_special_cases():
    rng = np.random.default_rng(9)
    V, gam, T = 40, 4, 0.7
    L = rng.standard_normal((gam + 1, V)) * 2.0
    spine = rng.integers(0, V, gam + 1)
    # q == p: every draft is accepted (u < 1 = p / q), and the bonus is drawn from p_gamma
    for seed in range(50):
        r, bonus, info = O.verify_sampled(L, L[:gam] / T, spine, T, seed, 0)
        assert r == gam
        assert bonus == O.gumbel_argmax(O.log_softmax(L[gam] / T), seed, O.TAG_BONUS, 0, 0)[0]
    # the target is sure of token a after t_0, the draft is another token: rejected at once,
    # and the residual max(0, p_0 - q_1) sits on a
    a = (int(spine[1]) + 3) % V
    L2 = L.copy()
    L2[0, a] += 60.0
    for seed in range(50):
        r, bonus, _ = O.verify_sampled(L2, L[:gam] / T, spine, T, seed, 1)
        assert (r, bonus) == (0, a)
    # the drafter is sure of t_1 and the target gives it probability p: accepted with rate p
    S = L[:gam] / T
    S[0, int(spine[1])] += 60.0
    p1 = _softmax(L[0] / T)[int(spine[1])]
    n = 3000
    acc = sum(O.verify_sampled(L, S, spine, T, 5, k)[0] >= 1 for k in range(n))
    assert abs(acc / n - p1) <= 5 * np.sqrt(p1 * (1 - p1) / n) + 1 / n
