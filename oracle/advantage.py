"""Oracle GRPO group advantage and gradient filter (float32) — test infrastructure only.

* Sec. 3.3, Eq. (4): samples are partitioned into groups N_k of identical
  prompts; the advantage of sample n is r_n minus the mean reward of its
  group.  Eq. (3) is the single-path special case of one group holding all N
  samples.  Sec. 3.3 also names dividing by the standard deviation as a
  standard modification; the workloads here use (r - mean) / (std + eps).
* Sec. 3.3 also names leaving sample n's own reward out of its baseline (fewer
  samples, less bias): LOO mode, A_n = r_n - (S - r_n) / (G - 1) with S the
  group's reward sum; as the single-path estimate it is the one-group case.
* Sec. 3.5: samples whose advantage is small are dropped from the gradient
  update.  Reading: keep sample n iff |A_n| >= tau; the kept indices are
  reported in ascending order.  tau = 0.1 (Appendix A hyper-parameter table).
* Sec. 3.4 / the preemptive-sampling figure: each prompt is duplicated into a
  group, so group k holds samples kG .. kG+G-1.

Arithmetic (so that the GPU matches bit for bit): float32 throughout, every
operation rounded on its own; a group sum is a pairwise tree over the group
zero-padded to a power of two, adjacent pairs first:
    mean = S(r) / G;  d = r - mean;  var = S(d*d) / (G - ddof);
    std = sqrt(var) (0 when G - ddof <= 0);  A = d (MEAN_ONLY) or d / (std + eps);
    LOO: A = r - (S(r) - r) / (G - 1)   (G >= 2).

Pins (tests/test_oracle_advantage.py): closed-form values of toy groups,
the zero-sum property, numpy's mean/std (ddof 0 and 1) as library routines, the
single-path Eq. (3) as one group, the closed-form kept set and expected kept
fraction for binary rewards; for LOO the exact fractions of toy groups, the
identity A_LOO = G / (G - 1) (r - mean) in exact arithmetic, and r_0 - r_1 for
pairs.
"""
from __future__ import annotations

import numpy as np

MEAN_ONLY, STD_POP, STD_SAMPLE, LOO = 0, 1, 2, 3


def pairwise_sum(v: np.ndarray) -> np.float32:
    """Sum of a float32 vector as a pairwise tree: pad to 2^k with zeros, add adjacent pairs."""
    a = np.asarray(v, dtype=np.float32).copy()
    n = 1
    while n < a.size:
        n *= 2
    a = np.concatenate([a, np.zeros(n - a.size, dtype=np.float32)])
    while a.size > 1:
        a = a[0::2] + a[1::2]
    return a[0]


def group_advantage(r: np.ndarray, group: int, mode: int = STD_SAMPLE, eps: float = 1e-6) -> np.ndarray:
    """GRPO advantage of every sample, float32 [N] (N = n_groups * group)."""
    r = np.asarray(r, dtype=np.float32)
    assert r.size % group == 0
    out = np.empty_like(r)
    G = np.float32(group)
    if mode == LOO:
        assert group >= 2, "the leave-one-out baseline needs at least two samples"
        for g0 in range(0, r.size, group):
            rg = r[g0:g0 + group]
            out[g0:g0 + group] = rg - (pairwise_sum(rg) - rg) / np.float32(group - 1)
        return out
    ddof = {MEAN_ONLY: 0, STD_POP: 0, STD_SAMPLE: 1}[mode]
    for g0 in range(0, r.size, group):
        rg = r[g0:g0 + group]
        mu = pairwise_sum(rg) / G
        d = rg - mu
        if mode == MEAN_ONLY:
            out[g0:g0 + group] = d
            continue
        if group - ddof > 0:
            var = pairwise_sum(d * d) / np.float32(group - ddof)
            sd = np.sqrt(var)
        else:
            sd = np.float32(0.0)
        out[g0:g0 + group] = d / (sd + np.float32(eps))
    return out


def gradient_filter(adv: np.ndarray, tau: float) -> np.ndarray:
    """Ascending int32 indices of samples with |A| >= tau (the samples kept for backprop)."""
    a = np.asarray(adv, dtype=np.float32)
    return np.flatnonzero(np.abs(a) >= np.float32(tau)).astype(np.int32)
