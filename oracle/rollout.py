"""Oracle of a whole rollout with per-sample completion lengths — test infrastructure only.

Sec. 3.4 (preemptive sampling): every prompt of one large batch is duplicated
into a group of G samples and the whole batch is decoded by the policy
pi_theta, each sample drawing its trajectory token by token (Sec. 3 problem
statement, Eq. (1)).  App. A caps a completion at a maximum length.  A sample's
completion therefore has its own length T_n <= cap; in a real run the sampled
end-of-sequence token sets it, here it is drawn beforehand (Geometric(1/600)
capped at 2048 for the ragged workload; readings in the design notes), and the
sample stops once it has drawn T_n tokens.  This module writes that schedule
out plainly:

* :func:`live_rows` — the samples still generating token t: those with T_n > t,
  in ascending sample order (the batch starts in sample order and retiring
  rows never reorders the others);
* :func:`retire_step` — the step at which a sample draws its last token;
* :func:`live_compact` — one step of the row bookkeeping: after token ``step``
  of every live row is drawn, the rows that go on (another token is due and the
  token just drawn is not the end-of-sequence id) move to the next step with
  their position and step advanced by one, in their order;
* :func:`kv_pages` — the cache pages a set of samples holds: the G samples of
  a prompt share the prompt's full pages, every sample owns the rest (a partial
  last prompt page is copied per sample at the fork);
* :func:`rollout` — the tokens themselves: sample n (= prompt * G + j, its id)
  draws token t from softmax(logits / T) with the oracle sampler's noise keyed
  by (seed, n, t), the logits being the oracle decoder's next-token logits after
  its prompt and its own first t tokens; the first token comes from the
  prompt's last position.

Pins (tests/test_oracle_rollout.py): iterating :func:`live_compact` from the
full batch reproduces :func:`live_rows` at every step; live counts sum to the
total number of generated tokens; the mean completion length of the ragged
workload against the closed form of a capped geometric law; a cut budget gives
a prefix of the uncut trajectory; an all-zero model draws argmax of the noise
alone and an embedding-only model follows a closed-form chain (both computed
without the decoder); page counts of hand-worked fork / retire cases.
"""
from __future__ import annotations

import numpy as np

from . import model as om
from . import sampler as osm


def live_rows(budgets, t: int) -> np.ndarray:
    """Sample ids still generating token ``t`` (T_n > t), ascending."""
    b = np.asarray(budgets)
    return np.flatnonzero(b > t).astype(np.int32)


def retire_step(budgets) -> np.ndarray:
    """Step at which each sample draws its last token (T_n - 1)."""
    return np.asarray(budgets, dtype=np.int64) - 1


def live_compact(tok, slot, pos, step, uid, budget, eos_id: int = -1):
    """One step of live-row bookkeeping, written as a loop over the rows in order.

    Row b holds (tok, slot, pos, step, uid) after its token for ``step`` was drawn.
    It goes on iff step + 1 < budget[uid] and (eos_id < 0 or tok != eos_id); the rows
    that go on are returned in their order with pos and step advanced by one.
    Returns five int32 arrays of the kept rows.
    """
    out = ([], [], [], [], [])
    for b in range(len(tok)):
        more = int(step[b]) + 1 < int(budget[int(uid[b])])
        ended = eos_id >= 0 and int(tok[b]) == eos_id
        if more and not ended:
            out[0].append(int(tok[b]))
            out[1].append(int(slot[b]))
            out[2].append(int(pos[b]) + 1)
            out[3].append(int(step[b]) + 1)
            out[4].append(int(uid[b]))
    return tuple(np.array(a, dtype=np.int32) for a in out)


def kv_pages(prompt_len: int, page_size: int, group: int, fed) -> int:
    """Pages held by samples whose caches hold ``fed[n]`` positions (0: retired / released).

    Sample n = prompt * group + j.  The prompt's full pages (floor(P / page_size))
    are held once per prompt while any of its samples holds its cache; each
    holding sample owns ceil(fed / page_size) - floor(P / page_size) more pages
    (the copied partial prompt page and the pages of its generated positions).
    """
    fed = np.asarray(fed, dtype=np.int64)
    full = prompt_len // page_size
    held = fed > 0
    n_prompts = len(fed) // group
    shared = sum(full for p in range(n_prompts) if held[p * group:(p + 1) * group].any())
    own = int(sum(-(-int(f) // page_size) - full for f in fed[held]))
    return shared + own


def rollout(shape: dict, weights: dict, prompts: np.ndarray, group: int, gen_len: int, temperature: float,
            seed: int, budgets=None, follow: np.ndarray | None = None) -> dict:
    """Tokens of every sample of a preemptive-sampling rollout.

    prompts int [n_prompts, P]; sample n uses prompt n // group and id n.  Sample n
    draws budgets[n] tokens (gen_len when budgets is None), each with
    :func:`oracle.sampler.sample_row` on the float32-cast float64 logits of
    :func:`oracle.model.forward` after its prompt and its previous tokens.

    ``follow`` (int [N, >= max budget], optional): the prefix each logits vector is
    computed after is the prompt plus follow[n][:t] instead of the oracle's own
    earlier tokens (teacher forcing along another run's trajectory).  Where the
    oracle's own tokens equal ``follow`` this is the free-running rollout.

    Returns dict with
      tokens   int32 [N, gen_len], -1 past a sample's end;
      logprob  float64 [N, gen_len], log softmax(l / T) at the drawn token (NaN past the end);
      margin   float64 [N, gen_len], the gap between the largest and the second largest
               Gumbel score l_v / T + g_v (float64, same noise) at each drawn position:
               logits within margin / 2 of these (max norm) draw the same token
               (up to the float32 rounding of the scores);
      score_of function (n, t, v) -> float64 score, for checking another token's validity.
    """
    prompts = np.asarray(prompts)
    n_prompts, P = prompts.shape
    N = n_prompts * group
    b = np.full(N, gen_len, dtype=np.int64) if budgets is None else np.asarray(budgets, dtype=np.int64)
    if b.shape != (N,) or (b < 1).any() or (b > gen_len).any():
        raise ValueError("budgets must hold N values in [1, gen_len]")
    V = shape["vocab"]
    T = float(np.float32(temperature))
    toks = np.full((N, gen_len), -1, dtype=np.int32)
    lps = np.full((N, gen_len), np.nan)
    margin = np.full((N, gen_len), np.nan)
    scores = {}
    for n in range(N):
        prompt = prompts[n // group]
        own: list[int] = []
        logits_all = None
        if follow is not None:  # every position at once: the prefixes are fixed
            seq = np.concatenate([prompt, np.asarray(follow[n][:b[n] - 1], dtype=prompt.dtype)])
            logits_all = om.forward(shape, weights, seq, positions=np.arange(P - 1, P - 1 + b[n]))
        for t in range(int(b[n])):
            if logits_all is not None:
                l64 = logits_all[t]
            else:
                seq = np.concatenate([prompt, np.asarray(own, dtype=prompt.dtype)])
                l64 = om.forward(shape, weights, seq, positions=[len(seq) - 1])[0]
            tok, lp = osm.sample_row(l64.astype(np.float32), n, t, temperature, seed)
            own.append(tok)
            toks[n, t] = tok
            lps[n, t] = lp
            g = osm.noise(seed, n, t, V).astype(np.float64)
            s = l64 / T + g
            if V > 1:
                top2 = np.partition(s, V - 2)[V - 2:]
                margin[n, t] = top2[1] - top2[0]
            else:
                margin[n, t] = np.inf
            scores[(n, t)] = s
    return {"tokens": toks, "logprob": lps, "margin": margin,
            "score_of": lambda n, t, v: float(scores[(n, t)][v])}
