"""Pins for the oracle of ragged rollouts (oracle/rollout.py): the live-row schedule,
compaction, page accounting and the token chain of a whole rollout."""
import dataclasses

import numpy as np
import pytest

from oracle import model as om
from oracle import rollout as oro
from oracle import sampler as osm
from paper_2505_17218_amd import synth


def test_iterated_compaction_reproduces_live_rows():
    """Starting from the whole batch after token 0, applying the compaction step by step
    leaves exactly the samples with T_n > t, in ascending order, at every step t; the
    live counts sum to the number of generated tokens."""
    rng = np.random.default_rng(0)
    N, T, P = 96, 50, 37
    budgets = rng.integers(1, T + 1, N).astype(np.int32)
    budgets[[0, 5]] = 1
    budgets[[1, 95]] = T
    uid = np.arange(N, dtype=np.int32)
    rows = (rng.integers(0, 1000, N).astype(np.int32), uid.copy(), np.full(N, P - 1, np.int32),
            np.zeros(N, np.int32), uid.copy())
    total = N  # every sample draws token 0
    for t in range(T):
        rows = oro.live_compact(*rows, budgets)
        live = oro.live_rows(budgets, t + 1)
        np.testing.assert_array_equal(rows[4], live)
        np.testing.assert_array_equal(rows[1], live)            # slot = sample id here
        assert (rows[2] == P + t).all() and (rows[3] == t + 1).all()
        total += len(live)
        rows = (rng.integers(0, 1000, len(live)).astype(np.int32),) + rows[1:]
    assert len(rows[0]) == 0
    assert total == int(budgets.sum())
    assert sum(len(oro.live_rows(budgets, t)) for t in range(T)) == int(budgets.sum())
    np.testing.assert_array_equal(oro.retire_step(budgets), budgets - 1)


def test_compaction_end_of_sequence():
    """With an end-of-sequence id, a row that has just drawn it stops even with budget left."""
    tok = np.array([7, 3, 7, 9], np.int32)
    slot = np.array([10, 11, 12, 13], np.int32)
    pos = np.array([5, 6, 7, 8], np.int32)
    step = np.array([0, 0, 2, 3], np.int32)
    uid = np.array([0, 1, 2, 3], np.int32)
    budget = np.array([5, 5, 3, 5], np.int32)
    out = oro.live_compact(tok, slot, pos, step, uid, budget, eos_id=7)
    # row 0: EOS; row 1 goes on; row 2: EOS and out of budget; row 3 goes on
    np.testing.assert_array_equal(out[1], [11, 13])
    np.testing.assert_array_equal(out[2], [7, 9])
    np.testing.assert_array_equal(out[3], [1, 4])
    out = oro.live_compact(tok, slot, pos, step, uid, budget, eos_id=-1)
    np.testing.assert_array_equal(out[4], [0, 1, 3])        # row 2: step 2 + 1 == budget 3
    empty = oro.live_compact(*(np.zeros(0, np.int32),) * 5, budget)
    assert all(len(a) == 0 for a in empty)


def test_ragged_workload_lengths_closed_form():
    """Geometric(1/600) on {1, 2, ...} capped at 2048: E[T] = (1 - (1 - p)^2048) / p = 580.3 and
    P(T = 2048) = (1 - p)^2047 = 3.29%; the expected live count before step t is N (1 - p)^t.
    The ragged workload's budgets (4096 samples, seed 0) follow these within sampling error."""
    p, cap = 1 / 600, 2048
    mean = (1 - (1 - p) ** cap) / p
    assert abs(mean - 580.3) < 0.05
    big = synth.make_lengths(400_000, 600.0, cap, seed=7)
    sd = np.sqrt(big.var() / big.size)
    assert abs(big.mean() - mean) < 5 * sd
    at_cap = (1 - p) ** (cap - 1)
    assert abs((big == cap).mean() - at_cap) < 5 * np.sqrt(at_cap * (1 - at_cap) / big.size)
    assert big.min() >= 1 and big.max() == cap
    wl = synth.WORKLOADS["1.5b-ragged"]
    b = synth.make_lengths(wl.n_seqs, wl.ragged_mean, wl.gen_len, 0)
    for t in (1, 100, 342, 600, 1500, 2047):
        q = (1 - p) ** t
        n_live = len(oro.live_rows(b, t))
        assert abs(n_live - wl.n_seqs * q) < 5 * np.sqrt(wl.n_seqs * q * (1 - q)) + 1, (t, n_live)
    assert len(oro.live_rows(b, cap)) == 0


def test_kv_pages_hand_cases():
    # P = 40, page 32: one shared full page per prompt, one copied partial page per sample
    P, ps, G = 40, 32, 4
    fed = np.full(8, 40)
    assert oro.kv_pages(P, ps, G, fed) == 2 * 1 + 8 * 1
    fed[0] = 65                                      # sample 0 grew into a third page
    assert oro.kv_pages(P, ps, G, fed) == 11
    fed[:4] = 0                                      # prompt 0's samples all retired
    assert oro.kv_pages(P, ps, G, fed) == 1 + 4
    fed[4:7] = 0                                     # one sample of prompt 1 still holds the shared page
    assert oro.kv_pages(P, ps, G, fed) == 1 + 1
    assert oro.kv_pages(P, ps, G, np.zeros(8)) == 0
    # P = 64 fills two pages: nothing is copied at the fork
    assert oro.kv_pages(64, 32, 8, np.full(16, 64)) == 2 * 2
    assert oro.kv_pages(64, 32, 8, np.full(16, 65)) == 2 * 2 + 16


MICRO = synth.Shape("micro-ro", 2, 16, 4, 2, 4, 24, 40, 10000.0, synth.DT_F32)


@pytest.fixture(scope="module")
def micro():
    w = synth.make_weights(MICRO, seed=21)
    for k in w:  # O(1) logits: tokens depend on the model, not on the noise alone
        if w[k].size and not k.endswith("norm"):
            w[k] = (w[k] * 40).astype(np.float32)
    prompts = np.random.default_rng(3).integers(0, MICRO.vocab, (3, 5)).astype(np.int32)
    return dataclasses.asdict(MICRO), w, prompts


def test_cut_budget_is_prefix_and_follow_is_free_running(micro):
    """A sample whose budget is cut draws the first tokens of its uncut trajectory and then
    nothing; teacher forcing along the free-running trajectory reproduces it exactly."""
    shape, w, prompts = micro
    G, T = 2, 9
    full = oro.rollout(shape, w, prompts, G, T, 1.0, 5)
    budgets = np.array([1, 9, 4, 2, 7, 3])
    cut = oro.rollout(shape, w, prompts, G, T, 1.0, 5, budgets=budgets)
    for n, b in enumerate(budgets):
        np.testing.assert_array_equal(cut["tokens"][n, :b], full["tokens"][n, :b])
        assert (cut["tokens"][n, b:] == -1).all() and np.isnan(cut["logprob"][n, b:]).all()
    fol = oro.rollout(shape, w, prompts, G, T, 1.0, 5, follow=full["tokens"])
    np.testing.assert_array_equal(fol["tokens"], full["tokens"])
    np.testing.assert_allclose(fol["logprob"], full["logprob"], rtol=0, atol=1e-12)
    assert (full["margin"] > 0).all()
    # samples of one prompt share the prompt but not the noise
    assert (full["tokens"][0] != full["tokens"][1]).any()


def test_zero_model_draws_argmax_of_the_noise(micro):
    """With every weight zero the logits vanish, so token t of sample n is the argmax of
    the noise keyed by (seed, n, t) alone, and every log-prob is -ln V."""
    shape, w, prompts = micro
    z = {k: np.zeros_like(v) for k, v in w.items()}
    G, T, seed = 2, 6, 11
    out = oro.rollout(shape, z, prompts, G, T, 1.0, seed)
    V = shape["vocab"]
    for n in range(prompts.shape[0] * G):
        for t in range(T):
            assert out["tokens"][n, t] == int(np.argmax(osm.noise(seed, n, t, V))), (n, t)
    np.testing.assert_allclose(out["logprob"], -np.log(V), rtol=0, atol=1e-12)


def test_embedding_only_model_chain(micro):
    """With the attention output and MLP down projections zero, the residual stream stays
    E[token], so the logits after a token are RMSNorm(E[token]) E^T: token 0 follows the
    prompt's last token, token t the sample's own token t - 1 (computed here without the
    decoder)."""
    shape, w, prompts = micro
    w2 = dict(w)
    for l in range(shape["n_layers"]):
        w2[f"l{l}.w_o"] = np.zeros_like(w[f"l{l}.w_o"])
        w2[f"l{l}.w_down"] = np.zeros_like(w[f"l{l}.w_down"])
    E = w2["embed"].astype(np.float64)
    g = w2["final_norm"].astype(np.float64)
    eps = shape["rms_eps"]

    def next_logits(tok):
        e = E[tok]
        return (e / np.sqrt(np.mean(e * e) + eps) * g) @ E.T

    G, T, seed, temp = 2, 7, 4, 0.7
    out = oro.rollout(shape, w2, prompts, G, T, temp, seed)
    for n in range(prompts.shape[0] * G):
        prev = int(prompts[n // G][-1])
        for t in range(T):
            tok, _ = osm.sample_row(next_logits(prev).astype(np.float32), n, t, temp, seed)
            assert out["tokens"][n, t] == tok, (n, t)
            prev = tok


def test_rollout_uses_the_decoder_logits(micro):
    """Token t of sample n is drawn from the decoder's logits after the prompt and the
    sample's first t tokens (the oracle forward pass, itself pinned in test_oracle_model)."""
    shape, w, prompts = micro
    G, T = 2, 5
    out = oro.rollout(shape, w, prompts, G, T, 1.0, 9)
    for n in (0, 3, 5):
        seq = np.concatenate([prompts[n // G], out["tokens"][n]])
        lg = om.forward(shape, w, seq[:len(prompts[0]) + T - 1])
        for t in range(T):
            tok, lp = osm.sample_row(lg[len(prompts[0]) - 1 + t].astype(np.float32), n, t, 1.0, 9)
            assert tok == out["tokens"][n, t]
            assert abs(lp - out["logprob"][n, t]) < 1e-12
