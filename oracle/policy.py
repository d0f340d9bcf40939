"""Oracle KL regulariser and PPO-style surrogate losses over the kept samples
(float64) — test infrastructure only.

* Sec. 3.2: PPO freezes the sampling policy pi_old and weights the gradient of
  pi_theta(y_n | x_n) by 1 / pi_old(y_n | x_n): a ratio of whole-trajectory
  probabilities, rho_n = pi_theta(y_n | x_n) / pi_old(y_n | x_n) =
  exp(S_n - S_old,n) with S = sum_t log pi(y_t | x, y_<t).  PPO clips for
  stability; reading: the clipped surrogate min(rho A, clip(rho, 1 - eps,
  1 + eps) A).  At theta = theta_old (rho = 1) its gradient is the PG gradient,
  as Sec. 3.2 notes.
* Sec. 3.2: the KL regulariser is the divergence D_KL(pi_base || pi_theta) from
  the original model, in that order.  Reading: along the sampled trajectory,
  the sum over generated positions of the exact KL between the two next-token
  distributions at that position (temperature 1), evaluated over the whole
  vocabulary; the reverse direction D_KL(pi_theta || pi_base) is reported beside
  it.  Entries whose logit is -inf have probability 0.
* Sec. 3.2: the regulariser enters with weight beta (J = J^PG or J^PPO plus
  beta J^KL); as a loss to minimise it is added, so the regularised loss is
      loss = -(1/N) sum_{n kept} surrogate_n + (beta/N) sum_{n kept} KL_n,
  with surrogate_n = A_n S_n (PG, no old policy) or the clipped PPO term.  The
  paper prints neither beta nor eps (its trainer keeps its defaults): both are
  arguments.  Sec. 3.5: only kept samples enter, still divided by N.
* Per kept sample the oracle also reports w_n = d loss / d S_n, the weight a
  backward pass puts on grad S_n: -A_n / N for PG; -A_n rho_n / N for PPO
  when the unclipped term is the minimum (ties included), else 0.

Pins (tests/test_oracle_policy.py): the KL of two-entry rows against the
Bernoulli closed form (asymmetric, so a swapped direction fails), scipy's
relative entropy on softmax rows as a library routine, zero for identical rows,
invariance under shifting a row by a constant, the closed form for a uniform
base row, -ln V - mean_v log p_theta(v); the teacher-forced KL vanishing for identical
models and obeying causality (a position's KL does not depend on later
tokens, nor on the last completion token at all); the PPO toy batch of exact
values on a dyadic grid covering both clipping sides and both advantage signs,
and rho = 1 giving the PG weights.
"""
from __future__ import annotations

import numpy as np

from . import model as om


def _log_softmax(x: np.ndarray) -> np.ndarray:
    """Row-wise log-softmax of float64 logits; -inf entries stay -inf."""
    x = np.asarray(x, dtype=np.float64)
    m = np.max(x, axis=-1, keepdims=True)
    return x - (m + np.log(np.sum(np.exp(x - m), axis=-1, keepdims=True)))


def kl_rows(theta_logits: np.ndarray, base_logits: np.ndarray) -> tuple[np.ndarray, np.ndarray]:
    """Exact KL of every row pair: (D_KL(p_base || p_theta), D_KL(p_theta || p_base)), float64 [R]."""
    la = _log_softmax(np.atleast_2d(theta_logits))
    lb = _log_softmax(np.atleast_2d(base_logits))
    pa, pb = np.exp(la), np.exp(lb)

    def kl(p, lp, lq):
        # sum over the entries p > 0 of p (log p - log q); log q = -inf there gives +inf
        out = np.zeros(p.shape[0])
        for r in range(p.shape[0]):
            s = p[r] > 0
            out[r] = np.sum(p[r, s] * (lp[r, s] - lq[r, s]))
        return out

    return kl(pb, lb, la), kl(pa, la, lb)


def teacher_forced_kl(shape: dict, w_theta: dict, w_base: dict, prompt: np.ndarray, completion: np.ndarray):
    """(lp_theta [T], kl [T], kl_rev [T]) along one sampled completion, float64.

    Row t compares the next-token distributions of the two models after the
    prompt and completion[:t] (the position that predicts completion[t]).
    """
    completion = np.asarray(completion)
    la = om.rollout_logits(shape, w_theta, prompt, completion)  # [T, V]
    lb = om.rollout_logits(shape, w_base, prompt, completion)
    lp = _log_softmax(la)[np.arange(completion.size), completion]
    kl, kl_rev = kl_rows(la, lb)
    return lp, kl, kl_rev


def policy_loss(lp: np.ndarray, adv: np.ndarray, kept: np.ndarray, lengths: np.ndarray | None = None,
                lp_old: np.ndarray | None = None, kl: np.ndarray | None = None, clip_eps: float = 0.2,
                beta: float = 0.0):
    """(loss, stats [N, 4]) over the kept samples, float64.

    stats[n] = (S_n, S_old_n, KL_n, w_n) for kept n (zeros elsewhere); without
    lp_old, S_old_n = S_n and the surrogate is A_n S_n (PG); without kl, KL_n = 0.
    """
    lp = np.asarray(lp, dtype=np.float64)
    N, T = lp.shape
    lens = np.full(N, T) if lengths is None else np.clip(np.asarray(lengths), 0, T)
    adv = np.asarray(adv, dtype=np.float64)
    stats = np.zeros((N, 4))
    sur_sum = 0.0
    kl_sum = 0.0
    for n in np.asarray(kept, dtype=np.int64):
        L = lens[n]
        S = float(np.sum(lp[n, :L]))
        S_old = float(np.sum(np.asarray(lp_old, dtype=np.float64)[n, :L])) if lp_old is not None else S
        K = float(np.sum(np.asarray(kl, dtype=np.float64)[n, :L])) if kl is not None else 0.0
        A = adv[n]
        if lp_old is None:
            sur = A * S
            w = -A / N
        else:
            rho = np.exp(S - S_old)
            unclipped = rho * A
            clipped = min(max(rho, 1.0 - clip_eps), 1.0 + clip_eps) * A
            sur = min(unclipped, clipped)
            w = -A * rho / N if unclipped <= clipped else 0.0
        stats[n] = (S, S_old, K, w)
        sur_sum += sur
        kl_sum += K
    loss = -sur_sum / N + beta * kl_sum / N
    return loss, stats
