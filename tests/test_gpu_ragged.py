"""Ragged rollouts (per-sample completion lengths; Sec. 3.4 preemptive sampling, App. A
maximum completion length) on the GPU against the oracle of oracle/rollout.py:

* the native driver's tokens against the oracle's rollout along the same trajectories:
  bit-exact wherever the oracle's best Gumbel score leads the runner-up by more than the
  logits tolerance allows to change, a valid draw (score within that tolerance of the
  best) elsewhere; exactly T_n tokens per sample and -1 after;
* a step-by-step ragged run through the C ABI (decode step, sampler, row compaction,
  release) whose live rows, their order and the pages the cache holds match the oracle's
  schedule at every step;
* the ragged workload itself (4096 samples, lengths Geometric(1/600) capped at 2048) at
  full size: structure exactly, sampled positions against the oracle, and the kept set of
  the gradient filter."""
import numpy as np
import pytest
import torch

from oracle import advantage as oa
from oracle import model as om
from oracle import rollout as oro
from oracle import sampler as osm
from paper_2505_17218_amd import _lib as L
from paper_2505_17218_amd import engine, synth

from gpu_util import dev_i32, make_kv, require_gpu, shape_dict

pytestmark = pytest.mark.gpu

TOL = {synth.DT_F32: 1e-4, synth.DT_BF16: 3e-2}
BF16_R = synth.Shape("bf16-ragged", 2, 256, 8, 2, 64, 512, 1000, 1e6, synth.DT_BF16)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def _check_against_oracle(shape, w, prompts, G, T, budgets, toks, lps, seed, tol):
    """GPU tokens / log-probs of a ragged rollout against oracle.rollout along them."""
    N = prompts.shape[0] * G
    ref = oro.rollout(shape_dict(shape), w, prompts, G, T, 1.0, seed, budgets=budgets, follow=toks)
    # structure: exactly budget tokens, -1 after (the oracle's schedule)
    for n in range(N):
        b = int(budgets[n])
        assert (toks[n, :b] >= 0).all() and (toks[n, :b] < shape.vocab).all(), n
        assert (toks[n, b:] == -1).all(), n
    np.testing.assert_array_equal(toks < 0, ref["tokens"] < 0)
    certified = ref["margin"] > 2 * tol + 1e-5
    live = ref["tokens"] >= 0
    np.testing.assert_array_equal(toks[certified & live], ref["tokens"][certified & live])
    for n, t in zip(*np.nonzero(live & ~certified)):
        best = ref["score_of"](n, t, int(ref["tokens"][n, t]))
        assert ref["score_of"](n, t, int(toks[n, t])) >= best - 2 * tol - 1e-5, (n, t)
    np.testing.assert_allclose(lps[live], ref["logprob"][live], rtol=0, atol=2 * tol + 5e-5)
    return int(certified[live].sum()), int(live.sum())


@pytest.mark.parametrize("shape_name", ["tiny", "bf16"])
def test_ragged_driver_matches_oracle(shape_name):
    """dash_rollout with budgets (rows at budget 1 and at the full length among them),
    eager and against the oracle; every page is back in the pool afterwards."""
    if shape_name == "tiny":
        wl = synth.WORKLOADS["tiny"]
        shape, n_prompts, G, P, T, ps = wl.shape, wl.n_prompts, wl.group, wl.prompt_len, wl.gen_len, 16
        w = synth.make_weights(shape, 0)
        prompts = synth.make_prompts(wl, 0)
    else:
        shape, n_prompts, G, P, T, ps = BF16_R, 3, 4, 45, 24, 32
        w = synth.make_weights(shape, 6)
        prompts = synth.make_prompts(synth.Workload("t", shape, n_prompts, G, P, T), 6)
    N = n_prompts * G
    budgets = np.random.default_rng(4).integers(1, T + 1, N).astype(np.int32)
    budgets[0], budgets[1], budgets[N - 1] = 1, T, 2
    model = engine.Model(shape, w)
    kv = make_kv(model, ps, N, P + T)
    total = kv.free_pages
    ro = engine.Rollout(model, kv, n_prompts, P, G, T)
    seed = 23
    toks, lps = ro.run(dev_i32(prompts), 1.0, seed, budgets=budgets, use_graph=False)
    torch.cuda.synchronize()
    toks, lps = toks.cpu().numpy(), lps.cpu().numpy()
    cert, n_tok = _check_against_oracle(shape, w, prompts, G, T, budgets, toks, lps, seed, TOL[shape.dtype])
    assert n_tok == int(budgets.sum())
    assert kv.free_pages == total
    assert L.dash_kv_device_status(kv.handle, engine.stream_handle()) == 0
    print(f"{shape_name}: {cert} of {n_tok} tokens certified bit-exact, the rest valid draws")


def test_ragged_stepwise_schedule_and_pages():
    """A ragged rollout driven step by step through the C ABI: after every step the live rows
    (from dash_live_compact) are the oracle's live set in order, and the pages the cache holds
    are exactly what the oracle's page accounting says for the positions each live sample has
    fed (shared prompt pages once per group while any of its samples lives).  The tokens equal
    the native driver's for the same budgets, bit for bit."""
    shape, n_prompts, G, P, T, ps = BF16_R, 3, 4, 45, 20, 32
    w = synth.make_weights(shape, 7)
    prompts = synth.make_prompts(synth.Workload("t", shape, n_prompts, G, P, T), 7)
    N = n_prompts * G
    budgets = np.random.default_rng(8).integers(1, T + 1, N).astype(np.int32)
    budgets[[0, 5]] = 1
    budgets[[1, 11]] = T
    model = engine.Model(shape, w)
    kv = make_kv(model, ps, N, P + T)
    total = kv.free_pages
    seed = 31
    st = engine.stream_handle()
    d_budget = dev_i32(budgets)
    logits0 = engine.prefill(model, kv, dev_i32(prompts), G, list(range(N)))
    fed = np.full(N, P)
    assert total - kv.free_pages == oro.kv_pages(P, ps, G, fed)
    uid = dev_i32(np.arange(N))
    tok, _ = engine.sample(logits0, uid, dev_i32(np.zeros(N)), 1.0, seed, row_of=dev_i32(np.arange(N) // G))
    toks = np.full((N, T), -1, np.int32)
    toks[:, 0] = tok.cpu().numpy()
    rows = [tok, dev_i32(np.arange(N)), dev_i32(np.full(N, P - 1)), dev_i32(np.zeros(N)), uid]
    ws = model.workspace(N, kv.max_ctx)
    for t in range(0, T):
        # compact after token t, then release the samples that drew their last token
        n = rows[0].numel()
        outs = [torch.empty(max(n, 1), dtype=torch.int32, device="cuda") for _ in range(5)]
        cnt = torch.zeros(1, dtype=torch.int32, device="cuda")
        L.dash_live_compact(*[r.data_ptr() for r in rows], d_budget.data_ptr(), -1, n,
                            *[o.data_ptr() for o in outs], cnt.data_ptr(), st)
        k = int(cnt.item())
        rows = [o[:k] for o in outs]
        live = oro.live_rows(budgets, t + 1)
        np.testing.assert_array_equal(rows[4].cpu().numpy(), live)
        done = np.flatnonzero(oro.retire_step(budgets) == t)
        L.dash_kv_release(kv.handle, done.tolist())
        fed[done] = 0
        assert total - kv.free_pages == oro.kv_pages(P, ps, G, fed), t
        if k == 0:
            break
        # next token: feed token t of every live row at position P + t
        L.dash_kv_reserve(kv.handle, live.tolist(), P + t + 1, st)
        fed[live] = P + t + 1
        assert total - kv.free_pages == oro.kv_pages(P, ps, G, fed), t
        logits = engine.decode_step(model, kv, rows[0], rows[1], rows[2], ws=ws)
        tok, _ = engine.sample(logits, rows[4], rows[3], 1.0, seed)
        toks[live, t + 1] = tok.cpu().numpy()
        rows[0] = tok
    assert kv.free_pages == total
    ro = engine.Rollout(model, kv, n_prompts, P, G, T)
    drv, _ = ro.run(dev_i32(prompts), 1.0, seed, budgets=budgets, use_graph=False)
    np.testing.assert_array_equal(drv.cpu().numpy(), toks)
    for n in range(N):
        assert (toks[n, budgets[n]:] == -1).all() and (toks[n, :budgets[n]] >= 0).all()


def test_ragged_workload_full_size():
    """The ragged workload at full size (1.5B shape, 512 prompts x 8 = 4096 samples, prompt
    256, lengths Geometric(1/600) capped at 2048): every sample draws exactly its budget,
    every page returns to the pool, sampled positions of the shortest, a capped and a typical
    sample are valid draws under the oracle's logits with log-probs within the tolerance, and
    the gradient filter's kept set equals the oracle's for the workload's rewards."""
    wl = synth.WORKLOADS["1.5b-ragged"]
    s = wl.shape
    N, P, T, ps = wl.n_seqs, wl.prompt_len, wl.gen_len, 32
    budgets = synth.make_lengths(N, wl.ragged_mean, T, 0)
    weights = synth.make_weights(s, 0)
    prompts = synth.make_prompts(wl, 0)
    model = engine.Model(s, weights)
    pages = wl.n_prompts * (P // ps) + int(sum((P + int(b) + ps - 1) // ps - P // ps for b in budgets)) + 8
    kv = engine.KVCache(model, ps, N, P + T, pages)
    total = kv.free_pages
    ro = engine.Rollout(model, kv, wl.n_prompts, P, wl.group, T)
    seed = synth.sampler_seed(0)
    toks, lps = ro.run(torch.from_numpy(prompts).cuda(), wl.temperature, seed, budgets=budgets)
    torch.cuda.synchronize()
    toks, lps = toks.cpu().numpy(), lps.cpu().numpy()
    assert kv.free_pages == total
    assert L.dash_kv_device_status(kv.handle, engine.stream_handle()) == 0
    lens = (toks >= 0).sum(axis=1)
    np.testing.assert_array_equal(lens, budgets)
    for n in range(N):
        assert (toks[n, budgets[n]:] == -1).all()
    assert (toks[toks >= 0] < s.vocab).all() and np.isfinite(lps[toks >= 0]).all()
    tol = TOL[s.dtype]
    shortest = int(np.argmin(budgets))
    capped = int(np.flatnonzero(budgets == T)[0])
    typical = int(np.argmin(np.abs(budgets - 600)))
    for n, ts in ((shortest, [0]), (typical, [0, 1, int(budgets[typical]) - 1]), (capped, [0, 700, T - 1])):
        ts = np.array([t for t in ts if t < budgets[n]])
        seq = np.concatenate([prompts[n // wl.group], toks[n][:ts.max()]])
        ref = om.forward(shape_dict(s), weights, seq, positions=P - 1 + ts)
        for i, t in enumerate(ts):
            l64 = ref[i]
            lse = l64.max() + np.log(np.exp(l64 - l64.max()).sum())
            tok = int(toks[n, t])
            assert abs((l64[tok] - lse) - lps[n, t]) <= 2 * tol, (n, t)
            sc = l64 + osm.noise(seed, n, int(t), s.vocab).astype(np.float64)
            assert sc[tok] >= sc.max() - 2 * tol, (n, t)
    rewards = synth.make_rewards(wl.n_prompts, wl.group, wl.reward, 0)
    adv, kept = engine.advantage_filter(torch.from_numpy(rewards).cuda(), wl.group, L.DASH_ADV_STD_SAMPLE, 1e-6, wl.tau)
    want = oa.group_advantage(rewards, wl.group, oa.STD_SAMPLE, 1e-6)
    np.testing.assert_array_equal(adv.cpu().numpy().view(np.uint32), want.view(np.uint32))
    np.testing.assert_array_equal(kept.cpu().numpy(), oa.gradient_filter(want, wl.tau))
    frac = kept.numel() / N
    assert abs(frac - 0.60724) < 4 * 0.022, frac
    print(f"ragged full size: {int(budgets.sum())} tokens, kept fraction {frac:.4f}")
