"""Oracle log-probabilities of sampled completions and the policy-gradient loss
over the kept samples (float64) — test infrastructure only.

* Sec. 3.2, Eq. (2): the policy-gradient estimate weights the gradient of
  log pi_theta(y_n | x_n) by the advantage of sample n; the probability of a
  trajectory is the product of its per-token conditionals (as written out for
  the SFT objective of Sec. 3.1), so log pi(y | x) = sum_t log pi(y_t | x, y_<t).
  The 1/len(y_n) weight of early GRPO versions is left out, as Sec. 3.2 says
  later versions do.
* Sec. 3.3 supplies A_n; Sec. 3.5 drops the samples with small |A_n| (they
  contribute nothing), so the sum runs over the kept samples only, still
  divided by the number N of all samples (the 1/N of the gradient estimate).

    lp[n, t] = log softmax(teacher-forced logits at position P - 1 + t)[y_{n,t}]
    loss = -(1/N) sum_{n kept} A_n sum_{t < len_n} lp[n, t]

Pins (tests/test_oracle_pg.py): with every weight zero the logits vanish and
lp = -ln V exactly; with only the embedding nonzero every layer is the
identity on the residual stream and lp has a closed form in the embedding
alone (evaluated independently with numpy); the log-probs of all V candidate
tokens at a position sum to probability 1; the loss of a hand-computed toy
batch, and its invariances (A = 0 gives 0, linear in A, no 1/len).
"""
from __future__ import annotations

import numpy as np

from . import model as om


def teacher_forced_logprobs(shape: dict, weights: dict, prompt: np.ndarray, completion: np.ndarray) -> np.ndarray:
    """float64 [T]: log pi(completion[t] | prompt, completion[:t]) under the oracle decoder."""
    completion = np.asarray(completion)
    logits = om.rollout_logits(shape, weights, prompt, completion)  # [T, V], row t predicts completion[t]
    m = logits.max(axis=1, keepdims=True)
    lse = m[:, 0] + np.log(np.exp(logits - m).sum(axis=1))
    return logits[np.arange(completion.size), completion] - lse


def pg_loss(lp: np.ndarray, adv: np.ndarray, kept: np.ndarray, lengths: np.ndarray | None = None):
    """(loss, sequence log-prob of every sample) over the kept samples, float64."""
    lp = np.asarray(lp, dtype=np.float64)
    N, T = lp.shape
    lens = np.full(N, T) if lengths is None else np.clip(np.asarray(lengths), 0, T)
    seq = np.array([lp[n, :lens[n]].sum() for n in range(N)])
    kept = np.asarray(kept, dtype=np.int64)
    loss = -float(np.sum(np.asarray(adv, dtype=np.float64)[kept] * seq[kept])) / N
    return loss, seq
