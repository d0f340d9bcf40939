"""Pins for the oracle teacher-forced log-probs and policy-gradient loss (oracle/pg.py)."""
import dataclasses

import numpy as np

from oracle import model as om
from oracle import pg
from paper_2505_17218_amd import synth

MICRO = synth.Shape("micro", 2, 16, 4, 2, 4, 24, 11, 1e4, synth.DT_F32)


def _sd(shape):
    return dataclasses.asdict(shape)


def _zero_weights(shape):
    w = synth.make_weights(shape, 0)
    return {k: np.zeros_like(v) for k, v in w.items()}


def test_zero_weights_give_uniform_log_probs():
    """All weights zero: every logit is 0, so every token has log-prob -ln V exactly."""
    w = _zero_weights(MICRO)
    for k in w:
        if "norm" in k:
            w[k] = np.ones_like(w[k])
    lp = pg.teacher_forced_logprobs(_sd(MICRO), w, np.array([1, 2, 3]), np.array([4, 0, 10, 7]))
    np.testing.assert_allclose(lp, -np.log(MICRO.vocab), rtol=0, atol=1e-12)


def test_embedding_only_closed_form():
    """Only the (tied) embedding nonzero: attention and MLP add zero, so the logits at a
    position are RMSNorm(E[token]) . E^T of that position's own token."""
    full = synth.make_weights(MICRO, 3)
    w = _zero_weights(MICRO)
    for k in w:
        if "norm" in k:
            w[k] = np.ones_like(w[k])
    w["embed"] = full["embed"]
    E = np.asarray(full["embed"], dtype=np.float64)
    prompt, comp = np.array([5, 1, 9]), np.array([2, 2, 8, 0, 3])
    got = pg.teacher_forced_logprobs(_sd(MICRO), w, prompt, comp)
    seq = np.concatenate([prompt, comp])
    P = prompt.size
    for t in range(comp.size):
        x = E[seq[P - 1 + t]]
        y = x / np.sqrt(np.mean(x * x) + MICRO.rms_eps)
        logits = E @ y
        want = logits[comp[t]] - (logits.max() + np.log(np.exp(logits - logits.max()).sum()))
        assert abs(got[t] - want) < 1e-10


def test_log_probs_normalise():
    """The log-probs of every candidate next token at one position sum to probability 1."""
    w = synth.make_weights(MICRO, 5)
    prompt = np.array([3, 1, 4, 1])
    total = 0.0
    for v in range(MICRO.vocab):
        total += np.exp(pg.teacher_forced_logprobs(_sd(MICRO), w, prompt, np.array([v]))[0])
    assert abs(total - 1.0) < 1e-12


def test_pg_loss_toy_and_invariances():
    lp = np.array([[-1.0, -2.0], [-0.5, -0.5], [-3.0, 0.0]])
    adv = np.array([1.0, -2.0, 0.5])
    # kept {0, 1}: -(1/3) (1 * -3 + -2 * -1) = 1/3
    loss, seq = pg.pg_loss(lp, adv, np.array([0, 1]))
    assert abs(loss - 1.0 / 3.0) < 1e-15
    np.testing.assert_array_equal(seq, [-3.0, -1.0, -3.0])
    # sample 0 truncated to one token: -(1/3) (1 * -1 + 2) = -1/3
    loss, _ = pg.pg_loss(lp, adv, np.array([0, 1]), lengths=np.array([1, 2, 2]))
    assert abs(loss + 1.0 / 3.0) < 1e-15
    assert pg.pg_loss(lp, np.zeros(3), np.arange(3))[0] == 0.0
    assert abs(pg.pg_loss(lp, 3 * adv, np.arange(3))[0] - 3 * pg.pg_loss(lp, adv, np.arange(3))[0]) < 1e-14
    # no 1/len: a sample twice as long with the same per-token log-prob counts twice as much
    lp2 = np.full((2, 4), -1.0)
    l2, _ = pg.pg_loss(lp2, np.array([1.0, 1.0]), np.array([0, 1]), lengths=np.array([2, 4]))
    assert abs(l2 - 3.0) < 1e-15
