"""Pins for the oracle sampler (oracle/sampler.py)."""
import math
import os
import shutil
import subprocess

import numpy as np
import pytest
from scipy import stats

from oracle import sampler as osm

HERE = os.path.dirname(os.path.abspath(__file__))


@pytest.fixture(scope="module")
def rocrand_ref(tmp_path_factory):
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc) or not os.path.exists("/opt/rocm/include/rocrand/rocrand_kernel.h"):
        pytest.skip("rocRAND headers / hipcc not available")
    exe = str(tmp_path_factory.mktemp("rr") / "rr")
    subprocess.run([hipcc, "-O1", os.path.join(HERE, "rocrand_philox_ref.cpp"), "-o", exe],
                   check=True, capture_output=True, timeout=300)

    def run(seed, subseq, offset, count):
        out = subprocess.run([exe, str(seed), str(subseq), str(offset), str(count)],
                             check=True, capture_output=True, text=True).stdout.split()
        return np.array([int(x, 16) for x in out], dtype=np.uint32)
    return run


@pytest.mark.parametrize("seed,uid,step,v0", [
    (0, 0, 0, 0), (2, 0, 0, 0), (0x123456789ABCDEF0, 7, 3, 40), (2, 1023, 1023, 151932),
    (0xFFFFFFFFFFFFFFFF, 0xFFFFFFFF, 0x3FFFFFFF, 4 * 0xFFFFFFF0)])
def test_philox_matches_rocrand_host_engine(rocrand_ref, seed, uid, step, v0):
    """rocRAND's engine: key = seed split in 32-bit halves, counter words (z, w) =
    subsequence, counter words (x, y) = offset / 4, output word = offset % 4.  Our
    counter (v>>2, step, seq_uid, 0) is subsequence = seq_uid, offset = 4*(step<<32 | v>>2) + (v&3)
    (the offset is a 64-bit count of outputs, so the mapping needs step < 2^30)."""
    n = 64
    offset = 4 * ((step << 32) | (v0 >> 2)) + (v0 & 3)
    ref = rocrand_ref(seed, uid, offset, n)
    v = v0 + np.arange(n)
    ctr = np.zeros((n, 4), dtype=np.uint32)
    ctr[:, 0] = (v >> 2).astype(np.uint32)
    ctr[:, 1] = step
    ctr[:, 2] = uid
    got = osm.philox4x32_10(ctr, (seed & 0xFFFFFFFF, seed >> 32))[np.arange(n), v & 3]
    np.testing.assert_array_equal(got, ref)


def test_noise_uses_philox_words_in_order():
    g = osm.noise(5, 3, 2, 10)
    ctr = np.zeros((3, 4), dtype=np.uint32)
    ctr[:, 0] = np.arange(3)
    ctr[:, 1] = 2
    ctr[:, 2] = 3
    x = osm.philox4x32_10(ctr, (5, 0)).reshape(-1)[:10]
    np.testing.assert_array_equal(g, osm.gumbel_from_bits(x))


def _ulp_err(got, x):
    ref = np.log(x.astype(np.float64))
    ulp = np.spacing(np.abs(ref).astype(np.float32)).astype(np.float64)
    return np.abs(got.astype(np.float64) - ref) / ulp


def test_own_log_accuracy():
    rng = np.random.default_rng(0)
    xs = [rng.random(200000, dtype=np.float32) + np.float32(0.5),              # around 1
          np.exp(rng.uniform(-87, 88, 200000)).astype(np.float32),            # full normal range
          (np.arange(1, 1 << 16, dtype=np.float32) * np.float32(2.0 ** -24)),  # the smallest u values
          np.float32(1.0) - np.arange(1, 5000, dtype=np.float32) * np.float32(2.0 ** -24)]
    for x in xs:
        x = x[(x > 0) & np.isfinite(x) & (x >= np.finfo(np.float32).tiny)]
        got = osm.own_log(x)
        err = _ulp_err(got, x)
        # about 3 ulp at worst (the rounding of s = f/(2+f) and of the series terms)
        assert err.max() <= 3.0, err.max()


def test_own_log_special_values():
    assert osm.own_log(np.array([1.0], np.float32))[0] == 0.0
    for k in (-20, -1, 1, 5, 100):
        got = float(osm.own_log(np.array([2.0 ** k], np.float32))[0])
        assert abs(got - k * math.log(2)) <= 2 * np.spacing(np.float32(abs(k * math.log(2))))


def test_uniform_open_interval():
    x = np.array([0, 1, 255, 256, 0xFFFFFFFF, 0xFFFFFF00], dtype=np.uint32)
    u = osm.uniform_from_bits(x)
    assert (u > 0).all() and (u < 1).all()
    assert u[0] == np.float32(2.0 ** -24) and u[4] == np.float32(1 - 2.0 ** -24)


def test_gumbel_moments():
    g = np.concatenate([osm.noise(9, uid, 0, 50000) for uid in range(8)]).astype(np.float64)
    n = g.size
    assert abs(g.mean() - 0.5772156649) < 5 * math.sqrt(math.pi ** 2 / 6 / n)
    assert abs(g.var() - math.pi ** 2 / 6) < 0.03


def test_token_frequencies_follow_softmax():
    l = np.array([0.3, -1.0, 2.0, 0.0, 0.5, -0.2, 1.1, -3.0], dtype=np.float32)
    for T in (1.0, 0.7):
        n = 40000
        toks = np.array([osm.sample_row(l, 17, step, T, 123)[0] for step in range(n)])
        p = np.exp(l.astype(np.float64) / T)
        p /= p.sum()
        obs = np.bincount(toks, minlength=8)
        chi2 = ((obs - n * p) ** 2 / (n * p)).sum()
        assert stats.chi2.sf(chi2, df=7) > 1e-4, (T, chi2)


def test_constant_logits_uniform():
    l = np.zeros(5, dtype=np.float32)
    n = 20000
    toks = np.array([osm.sample_row(l, 1, s, 1.0, 7)[0] for s in range(n)])
    obs = np.bincount(toks, minlength=5)
    chi2 = ((obs - n / 5) ** 2 / (n / 5)).sum()
    assert stats.chi2.sf(chi2, df=4) > 1e-4


def test_small_temperature_is_argmax():
    rng = np.random.default_rng(4)
    l = rng.standard_normal(1000).astype(np.float32)
    for step in range(20):
        tok, lp = osm.sample_row(l, 3, step, 1e-4, 99)
        assert tok == int(np.argmax(l))
        assert abs(lp) < 1e-6 or lp > -1e-3


def test_logprob_normalised_and_nonfinite():
    rng = np.random.default_rng(5)
    l = rng.standard_normal(64).astype(np.float32) * 3
    T = 0.8
    z = l.astype(np.float64) / np.float64(np.float32(T))
    lps = z - (z.max() + np.log(np.exp(z - z.max()).sum()))
    assert abs(np.exp(lps).sum() - 1) < 1e-12
    tok, lp = osm.sample_row(l, 0, 0, T, 1)
    assert abs(lp - lps[tok]) < 1e-12
    l2 = l.copy()
    l2[[3, 10]] = [np.inf, np.nan]
    for s in range(50):
        t2, _ = osm.sample_row(l2, 0, s, 1.0, 1)
        assert t2 not in (3, 10)
    assert osm.sample_row(np.full(4, np.nan, np.float32), 0, 0, 1.0, 1)[0] == -1


def test_argmax_tie_lowest_index():
    s = np.array([1.0, 3.0, 2.0, 3.0], np.float32)
    assert osm.argmax_lowest(s, np.ones(4, bool)) == 1
    assert osm.argmax_lowest(s, np.array([True, False, True, True])) == 3
