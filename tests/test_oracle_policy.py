"""Pins for the oracle KL regulariser and PPO-style losses (oracle/policy.py)."""
import dataclasses

import numpy as np
import scipy.special
import scipy.stats

from oracle import policy
from paper_2505_17218_amd import synth

MICRO = synth.Shape("micro", 2, 16, 4, 2, 4, 24, 11, 1e4, synth.DT_F32)


def _sd(shape):
    return dataclasses.asdict(shape)


def test_kl_bernoulli_closed_form():
    """Two-entry rows are Bernoulli distributions: D_KL(Bern(p) || Bern(q)) =
    p ln(p/q) + (1-p) ln((1-p)/(1-q)).  p != q asymmetric, so a swapped direction fails."""
    for a0, a1, b0, b1 in [(0.3, -1.2, 2.0, 0.1), (5.0, -5.0, 0.0, 0.0), (-0.7, 0.4, 1.9, -2.6)]:
        # both masses of each distribution directly (1 - q would cancel for q near 1)
        q, q1 = np.exp(a0) / (np.exp(a0) + np.exp(a1)), np.exp(a1) / (np.exp(a0) + np.exp(a1))  # theta
        p, p1 = np.exp(b0) / (np.exp(b0) + np.exp(b1)), np.exp(b1) / (np.exp(b0) + np.exp(b1))  # base
        kl, kl_rev = policy.kl_rows(np.array([[a0, a1]]), np.array([[b0, b1]]))
        want = p * np.log(p / q) + p1 * np.log(p1 / q1)
        want_rev = q * np.log(q / p) + q1 * np.log(q1 / p1)
        assert abs(kl[0] - want) < 1e-14 and abs(kl_rev[0] - want_rev) < 1e-14
        assert abs(want - want_rev) > 1e-6  # far beyond the 1e-14 tolerance


def test_kl_matches_scipy_relative_entropy():
    """scipy.stats.entropy(pk, qk) is sum pk log(pk / qk): the library routine on softmax rows."""
    a = synth.make_logits(6, 97, seed=1, scale=2.0).astype(np.float64)
    b = synth.make_logits(6, 97, seed=2, scale=2.0).astype(np.float64)
    kl, kl_rev = policy.kl_rows(a, b)
    pa, pb = scipy.special.softmax(a, axis=1), scipy.special.softmax(b, axis=1)
    for r in range(6):
        assert abs(kl[r] - scipy.stats.entropy(pb[r], pa[r])) < 1e-12
        assert abs(kl_rev[r] - scipy.stats.entropy(pa[r], pb[r])) < 1e-12
        assert kl[r] > 0 and kl_rev[r] > 0


def test_kl_identical_rows_and_shift_invariance():
    a = synth.make_logits(4, 50, seed=3).astype(np.float64)
    kl, kl_rev = policy.kl_rows(a, a)
    assert np.all(kl == 0.0) and np.all(kl_rev == 0.0)
    b = synth.make_logits(4, 50, seed=4).astype(np.float64)
    k0, r0 = policy.kl_rows(a, b)
    k1, r1 = policy.kl_rows(a + 3.25, b - 7.5)
    np.testing.assert_allclose(k1, k0, rtol=0, atol=1e-13)
    np.testing.assert_allclose(r1, r0, rtol=0, atol=1e-13)


def test_kl_uniform_base_closed_form():
    """Constant base row (uniform p_base): D_KL(U || p_theta) = -ln V - mean_v log p_theta(v),
    and D_KL(p_theta || U) = ln V - H(p_theta)."""
    V = 40
    a = synth.make_logits(3, V, seed=5, scale=1.5).astype(np.float64)
    kl, kl_rev = policy.kl_rows(a, np.zeros((3, V)))
    for r in range(3):
        lsm = a[r] - scipy.special.logsumexp(a[r])
        assert abs(kl[r] - (-np.log(V) - lsm.mean())) < 1e-13
        assert abs(kl_rev[r] - (np.log(V) - scipy.stats.entropy(np.exp(lsm)))) < 1e-13


def test_kl_masked_entries():
    """-inf logits have probability 0: a base zero adds nothing, a theta zero under base mass is +inf."""
    a = np.array([[0.5, -np.inf, 1.0]])
    b = np.array([[0.2, -np.inf, -0.3]])
    kl, kl_rev = policy.kl_rows(a, b)
    kl2, kl2_rev = policy.kl_rows(a[:, [0, 2]], b[:, [0, 2]])
    assert abs(kl[0] - kl2[0]) < 1e-15 and abs(kl_rev[0] - kl2_rev[0]) < 1e-15
    kl, kl_rev = policy.kl_rows(np.array([[0.0, -np.inf]]), np.array([[0.0, 0.0]]))
    assert kl[0] == np.inf and abs(kl_rev[0] - np.log(2.0)) < 1e-15


def test_teacher_forced_kl_identical_models_and_causality():
    w = synth.make_weights(MICRO, 7)
    wb = synth.make_weights(MICRO, 8)
    prompt, comp = np.array([3, 1, 4]), np.array([1, 5, 9, 2, 6])
    lp, kl, kl_rev = policy.teacher_forced_kl(_sd(MICRO), w, w, prompt, comp)
    assert np.all(kl == 0.0) and np.all(kl_rev == 0.0)
    lp, kl, kl_rev = policy.teacher_forced_kl(_sd(MICRO), w, wb, prompt, comp)
    assert np.all(kl > 0) and np.all(kl_rev > 0)
    # the last completion token is only a target: no KL depends on it
    c2 = comp.copy()
    c2[-1] = (c2[-1] + 3) % MICRO.vocab
    _, kl2, _ = policy.teacher_forced_kl(_sd(MICRO), w, wb, prompt, c2)
    np.testing.assert_array_equal(kl2, kl)
    # changing completion token t changes the KL of later positions only
    t = 2
    c3 = comp.copy()
    c3[t] = (c3[t] + 1) % MICRO.vocab
    _, kl3, _ = policy.teacher_forced_kl(_sd(MICRO), w, wb, prompt, c3)
    np.testing.assert_array_equal(kl3[: t + 1], kl[: t + 1])
    assert np.all(kl3[t + 1:] != kl[t + 1:])


def test_policy_loss_pg_mode_matches_definition():
    """Without an old policy the surrogate is A_n S_n: loss and weights -A_n / N."""
    lp = np.array([[-1.0, -2.0], [-0.5, -0.5], [-3.0, 0.0]])
    adv = np.array([1.0, -2.0, 0.5])
    loss, st = policy.policy_loss(lp, adv, np.array([0, 1]))
    assert abs(loss - 1.0 / 3.0) < 1e-15
    np.testing.assert_array_equal(st[:, 0], [-3.0, -1.0, 0.0])
    np.testing.assert_array_equal(st[:, 3], [-1.0 / 3.0, 2.0 / 3.0, 0.0])
    kl = np.array([[0.25, 0.5], [0.125, 0.0], [9.0, 9.0]])
    loss_b, st_b = policy.policy_loss(lp, adv, np.array([0, 1]), kl=kl, beta=0.5)
    assert abs(loss_b - (1.0 / 3.0 + 0.5 * 0.875 / 3.0)) < 1e-15
    np.testing.assert_array_equal(st_b[:, 2], [0.75, 0.125, 0.0])


def test_policy_loss_ppo_clipping_toy():
    """Sequence ratios on a dyadic grid, eps = 0.25, N = 4, all kept:
    n0: rho = e^0 = 1, A = 1       -> surrogate 1, w = -1/4
    n1: rho = e^{ln 2} = 2, A = 1  -> clipped at 1.25: surrogate 1.25, w = 0
    n2: rho = 2, A = -1            -> min(-2, -1.25) = -2 unclipped, w = 2/4
    n3: rho = 1/2, A = -2          -> min(-1, -1.5) = -1.5 clipped, w = 0
    loss = -(1 + 1.25 - 2 - 1.5) / 4 = 0.3125."""
    ln2 = np.log(2.0)
    lp = np.array([[-1.0, 0.0], [-1.0, 0.0], [-1.0, 0.0], [-1.0, 0.0]])
    lp_old = np.array([[-1.0, 0.0], [-1.0 - ln2, 0.0], [-1.0 - ln2, 0.0], [-1.0 + ln2, 0.0]])
    adv = np.array([1.0, 1.0, -1.0, -2.0])
    loss, st = policy.policy_loss(lp, adv, np.arange(4), lp_old=lp_old, clip_eps=0.25)
    assert abs(loss - 0.3125) < 1e-14
    np.testing.assert_allclose(st[:, 3], [-0.25, 0.0, 0.5, 0.0], rtol=0, atol=1e-14)
    # rho = 1 everywhere: the weights are the PG weights -A_n / N (Sec. 3.2: PPO = PG at theta_old)
    _, st_pg = policy.policy_loss(lp, adv, np.arange(4))
    _, st_eq = policy.policy_loss(lp, adv, np.arange(4), lp_old=lp, clip_eps=0.25)
    np.testing.assert_array_equal(st_eq[:, 3], st_pg[:, 3])
    # lengths truncate every per-sample sum, the KL included
    kl = np.full((4, 2), 0.5)
    _, st_l = policy.policy_loss(lp, adv, np.arange(4), lengths=np.array([1, 2, 0, 2]), lp_old=lp_old, kl=kl)
    np.testing.assert_array_equal(st_l[:, 2], [0.5, 1.0, 0.0, 1.0])
