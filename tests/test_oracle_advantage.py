"""Pins for the oracle GRPO advantage and gradient filter (oracle/advantage.py)."""
import json
import math
import os

import numpy as np
import pytest

from oracle import advantage as oa
from paper_2505_17218_amd import synth

HERE = os.path.dirname(os.path.abspath(__file__))
MODES = {"MEAN_ONLY": oa.MEAN_ONLY, "STD_POP": oa.STD_POP, "STD_SAMPLE": oa.STD_SAMPLE}


def _golden():
    with open(os.path.join(HERE, "golden", "toy_advantage.json")) as f:
        return json.load(f)


@pytest.mark.parametrize("case", _golden()["cases"], ids=lambda c: f"{c['mode']}-G{c['G']}-{c['r']}")
def test_toy_groups_closed_form(case):
    eps = _golden()["eps"]
    r = np.array(case["r"], dtype=np.float32)
    mean = case["mean"][0] / case["mean"][1]
    want = r.astype(np.float64) - mean
    scale = 1.0
    if case["mode"] != "MEAN_ONLY":
        scale = math.sqrt(case["var"][0] / case["var"][1]) + eps
        want = want / scale
    got = oa.group_advantage(r, case["G"], MODES[case["mode"]], eps)
    # float32 evaluation of the closed form: a few ulp, plus the rounding of the
    # mean carried through r - mean (absolute, relative to max|r| / scale)
    atol = 8 * 2.0 ** -24 * np.abs(r).max() / scale
    np.testing.assert_allclose(got, want, rtol=4 * 2.0 ** -24, atol=atol)
    if case["mode"] == "MEAN_ONLY":
        np.testing.assert_array_equal(got, want.astype(np.float32))


def test_library_mean_std():
    rng = np.random.default_rng(0)
    for G in (1, 2, 3, 4, 5, 8, 16, 33, 64, 100):
        r = rng.standard_normal(7 * G).astype(np.float32)
        rg = r.reshape(7, G).astype(np.float64)
        d = rg - rg.mean(axis=1, keepdims=True)
        np.testing.assert_allclose(oa.group_advantage(r, G, oa.MEAN_ONLY).reshape(7, G), d, atol=1e-5)
        for mode, ddof in ((oa.STD_POP, 0), (oa.STD_SAMPLE, 1)):
            if G - ddof <= 0:
                sd = np.zeros((7, 1))
            else:
                sd = rg.std(axis=1, ddof=ddof, keepdims=True)
            want = d / (sd + 1e-6)
            got = oa.group_advantage(r, G, mode).reshape(7, G)
            np.testing.assert_allclose(got, want, rtol=2e-5, atol=1e-5)


def test_zero_sum_and_uniform_groups():
    r = synth.make_rewards(64, 8, "beta0.5", seed=1)
    a = oa.group_advantage(r, 8, oa.MEAN_ONLY).reshape(64, 8).astype(np.float64)
    assert (a.sum(axis=1) == 0).all()   # binary rewards, G = 2^k: every partial sum is exact
    s = oa.group_advantage(r, 8, oa.STD_SAMPLE).reshape(64, 8)
    uniform = (r.reshape(64, 8) == r.reshape(64, 8)[:, :1]).all(axis=1)
    assert (s[uniform] == 0).all() and not np.signbit(s[uniform]).any()


def test_single_path_is_one_group():
    """Eq. (3): the single-path advantage is the GRPO advantage with one group of all N."""
    r = np.random.default_rng(2).random(64).astype(np.float32)
    a = oa.group_advantage(r, 64, oa.MEAN_ONLY)
    np.testing.assert_allclose(a, r.astype(np.float64) - r.astype(np.float64).mean(), atol=1e-6)


def test_leave_one_out_toy_groups():
    """LOO baseline (Sec. 3.3): A_n = r_n - mean of the other samples, exact fractions."""
    got = oa.group_advantage(np.array([1, 0, 0, 0], np.float32), 4, oa.LOO)
    np.testing.assert_array_equal(got, np.array([1.0, -1 / 3, -1 / 3, -1 / 3], np.float32))
    # G = 8, rewards (1, 1, 0, 1, 0, 0, 0, 0): ones get 1 - 2/7, zeros get -3/7
    r = np.array([1, 1, 0, 1, 0, 0, 0, 0], np.float32)
    want = np.where(r == 1, 1 - 2 / 7, -3 / 7)
    np.testing.assert_allclose(oa.group_advantage(r, 8, oa.LOO), want, rtol=2 * 2.0 ** -24, atol=0)
    # pairs: the baseline is the other sample (rewards on a 2^-10 grid, so every sum is exact)
    r2 = (np.random.default_rng(3).integers(0, 1024, 40) / 1024).astype(np.float32)
    a2 = oa.group_advantage(r2, 2, oa.LOO).reshape(20, 2)
    rr = r2.reshape(20, 2)
    np.testing.assert_array_equal(a2[:, 0], rr[:, 0] - rr[:, 1])
    np.testing.assert_array_equal(a2[:, 1], rr[:, 1] - rr[:, 0])


def test_leave_one_out_is_scaled_mean_centering():
    """In exact arithmetic r - (S - r)/(G - 1) = G/(G - 1) (r - S/G); float32 within a few ulp."""
    rng = np.random.default_rng(4)
    for G in (2, 3, 5, 8, 100, 4096):
        r = rng.random(3 * G).astype(np.float32)
        rg = r.reshape(3, G).astype(np.float64)
        want = G / (G - 1) * (rg - rg.mean(axis=1, keepdims=True))
        got = oa.group_advantage(r, G, oa.LOO).reshape(3, G)
        np.testing.assert_allclose(got, want, atol=8 * G * 2.0 ** -24)


def test_pairwise_sum_order():
    v = np.array([1e8, 1.0, -1e8, 1.0], np.float32)
    # ((1e8 + 1) + (-1e8 + 1)) in float32 = 1e8 + -1e8 = 0
    assert oa.pairwise_sum(v) == np.float32(0.0)
    assert oa.pairwise_sum(np.array([1.0, 2.0, 3.0], np.float32)) == np.float32(6.0)


@pytest.mark.parametrize("G,mode", [(4, oa.MEAN_ONLY), (4, oa.STD_POP), (4, oa.STD_SAMPLE),
                                    (8, oa.MEAN_ONLY), (8, oa.STD_POP), (8, oa.STD_SAMPLE)])
def test_binary_rewards_keep_exactly_mixed_groups(G, mode):
    """For binary rewards the smallest nonzero |A| is 1/G (mean only), 1/sqrt(G-1) (population std)
    or 1/sqrt(G) (sample std); all exceed tau = 0.1 for G <= 9, so exactly the members of groups
    with mixed rewards are kept."""
    r = synth.make_rewards(500, G, "beta0.5", seed=3)
    kept = oa.gradient_filter(oa.group_advantage(r, G, mode), 0.1)
    rg = r.reshape(-1, G)
    mixed = ~(rg == rg[:, :1]).all(axis=1)
    want = np.flatnonzero(np.repeat(mixed, G)).astype(np.int32)
    np.testing.assert_array_equal(kept, want)
    assert (np.diff(kept) > 0).all()


def test_expected_kept_fraction_closed_form():
    """P(mixed group) = 1 - 2 E[p^G] with E[p^G] = prod_{i<G} (a+i)/(a+b+i) for p ~ Beta(a, b)."""
    for kind, G, n in (("bernoulli0.5", 4, 20000), ("beta0.5", 8, 20000), ("beta0.5", 4, 20000)):
        if kind == "bernoulli0.5":
            want = 1 - 2 * 0.5 ** G
        else:
            want = 1 - 2 * np.prod([(0.5 + i) / (1.0 + i) for i in range(G)])
        r = synth.make_rewards(n, G, kind, seed=4)
        frac = oa.gradient_filter(oa.group_advantage(r, G), 0.1).size / r.size
        se = math.sqrt(want * (1 - want) / n)
        assert abs(frac - want) < 5 * se, (kind, G, frac, want)


def test_filter_boundary_and_zero_threshold():
    a = np.array([0.1, -0.1, 0.099999994, 0.0, -0.0, 1e-45], np.float32)
    np.testing.assert_array_equal(oa.gradient_filter(a, 0.1), [0, 1])
    np.testing.assert_array_equal(oa.gradient_filter(a, np.float32(1e-45)), [0, 1, 2, 5])
