"""Full-size parity: the 1.5B-shaped workload of the benchmark (128 prompts x G = 8 =
1024 sequences, prompt 256, 1024 generated tokens, bf16, page size 32, the rollout
driver exactly as bench.py runs it), checked on sampled sequences and positions
against the oracle, plus properties that hold at any size."""
import numpy as np
import pytest
import torch

from oracle import model as om
from oracle import policy as opol
from oracle import sampler as osm
from paper_2505_17218_amd import engine, synth

from gpu_util import dev_i32, kl_sensitivity, require_gpu, shape_dict

pytestmark = pytest.mark.gpu

# logits within 3e-2 (bf16 tolerance) move a log-softmax value by at most 2 * 3e-2
LP_TOL = 6e-2
LOGIT_TOL = 3e-2


@pytest.fixture(scope="module")
def rollout_1p5b():
    require_gpu()
    wl = synth.WORKLOADS["1.5b-b1024"]
    s = wl.shape
    weights = synth.make_weights(s, 0)
    prompts = synth.make_prompts(wl, 0)
    model = engine.Model(s, weights)
    N, P, T, ps = wl.n_seqs, wl.prompt_len, wl.gen_len, 32
    pages = wl.n_prompts * (P // ps) + N * ((P + T + ps - 1) // ps - P // ps) + 8
    kv = engine.KVCache(model, ps, N, P + T, pages)
    ro = engine.Rollout(model, kv, wl.n_prompts, P, wl.group, T)
    seed = synth.sampler_seed(0)
    d_prompts = torch.from_numpy(prompts).cuda()
    toks, lps = ro.run(d_prompts, wl.temperature, seed, use_graph=False)
    torch.cuda.synchronize()
    toks, lps = toks.cpu().numpy().copy(), lps.cpu().numpy().copy()
    again, _ = ro.run(d_prompts, wl.temperature, seed, use_graph=False)
    torch.cuda.synchronize()
    return dict(wl=wl, weights=weights, prompts=prompts, toks=toks, lps=lps, again=again.cpu().numpy(), seed=seed,
                model=model, kv=kv)


def test_fullsize_properties(rollout_1p5b):
    r = rollout_1p5b
    V = r["wl"].shape.vocab
    toks, lps = r["toks"], r["lps"]
    assert toks.shape == (1024, 1024)
    assert ((toks >= 0) & (toks < V)).all()
    assert np.isfinite(lps).all() and (lps <= 1e-6).all()
    np.testing.assert_array_equal(toks, r["again"])  # bit-reproducible run to run
    # samples of one prompt share the prompt but draw independent noise: they diverge
    assert (toks[0] != toks[1]).any()


@pytest.mark.parametrize("n", [0, 777])
def test_fullsize_sampled_sequences_match_oracle(rollout_1p5b, n):
    r = rollout_1p5b
    wl = r["wl"]
    P, G = wl.prompt_len, wl.group
    ts = np.array([0, 1, 2, 31, 32, 255, 511, 1023])
    seq = np.concatenate([r["prompts"][n // G], r["toks"][n][:ts.max()]])
    ref = om.forward(shape_dict(wl.shape), r["weights"], seq, positions=P - 1 + ts)
    for i, t in enumerate(ts):
        l64 = ref[i]
        lse = l64.max() + np.log(np.exp(l64 - l64.max()).sum())
        tok = int(r["toks"][n, t])
        assert abs((l64[tok] - lse) - r["lps"][n, t]) <= LP_TOL, (n, t)
        # the GPU token is a valid Gumbel-max draw under the oracle's logits: its score is
        # within the logits tolerance of the best score for the same noise
        g = osm.noise(r["seed"], n, int(t), wl.shape.vocab).astype(np.float64)
        s = l64 + g
        assert s[tok] >= s.max() - 2 * LOGIT_TOL, (n, t)


def test_fullsize_teacher_forced_recompute(rollout_1p5b):
    """Teacher-forced log-probs of three full 1280-token sequences (prefill path, LM head
    over every completion position) reproduce the log-probs recorded while sampling bit
    for bit (the contexts fit the cache's single 2048-key attention split)."""
    r = rollout_1p5b
    wl = r["wl"]
    P, G = wl.prompt_len, wl.group
    ns = [0, 777, 1023]
    seqs = np.concatenate([r["prompts"][[n // G for n in ns]], r["toks"][ns]], axis=1).astype(np.int32)
    rec = engine.teacher_forced_logprobs(r["model"], r["kv"], torch.from_numpy(seqs).cuda(), P).cpu().numpy()
    assert np.isfinite(rec).all()
    assert P + wl.gen_len <= r["kv"].split_keys
    np.testing.assert_array_equal(rec.view(np.uint32), r["lps"][ns].view(np.uint32))


@pytest.mark.parametrize("workload,ns,ts", [("0.5b-b512", [0, 301, 511], [0, 1, 255, 1023]),
                                            ("3b-b64", [0, 63], [0, 511, 1023])])
def test_other_workloads_sampled_against_oracle(workload, ns, ts):
    """The 0.5B (512 sequences) and 3B (64 sequences, prompt 512) workloads at full size:
    sampled positions of sampled sequences against the oracle, as for the 1.5B run."""
    require_gpu()
    wl = synth.WORKLOADS[workload]
    s = wl.shape
    weights = synth.make_weights(s, 0)
    prompts = synth.make_prompts(wl, 0)
    model = engine.Model(s, weights)
    N, P, T, ps = wl.n_seqs, wl.prompt_len, wl.gen_len, 32
    pages = wl.n_prompts * (P // ps) + N * ((P + T + ps - 1) // ps - P // ps) + 8
    kv = engine.KVCache(model, ps, N, P + T, pages)
    ro = engine.Rollout(model, kv, wl.n_prompts, P, wl.group, T)
    seed = synth.sampler_seed(0)
    toks, lps = ro.run(torch.from_numpy(prompts).cuda(), wl.temperature, seed)
    torch.cuda.synchronize()
    toks, lps = toks.cpu().numpy(), lps.cpu().numpy()
    assert ((toks >= 0) & (toks < s.vocab)).all() and np.isfinite(lps).all()
    ts = np.array(ts)
    for n in ns:
        seq = np.concatenate([prompts[n // wl.group], toks[n][:ts.max()]])
        ref = om.forward(shape_dict(s), weights, seq, positions=P - 1 + ts)
        for i, t in enumerate(ts):
            l64 = ref[i]
            lse = l64.max() + np.log(np.exp(l64 - l64.max()).sum())
            tok = int(toks[n, t])
            assert abs((l64[tok] - lse) - lps[n, t]) <= LP_TOL, (workload, n, t)
            g = osm.noise(seed, n, int(t), s.vocab).astype(np.float64)
            sc = l64 + g
            assert sc[tok] >= sc.max() - 2 * LOGIT_TOL, (workload, n, t)


def test_fullsize_teacher_forced_kl(rollout_1p5b):
    """KL(base || policy) and its reverse along a sampled 1.5B-shape sequence (V = 151,936)
    against an independently initialised base model of the same shape: sampled positions
    against the oracle, within the first-order effect of the bf16 logits tolerance (twice the
    bound plus 4 delta^2); the policy's log-probs equal the ones recorded while sampling."""
    r = rollout_1p5b
    wl = r["wl"]
    s, P, n, T = wl.shape, wl.prompt_len, 13, 40
    base_w = synth.make_weights(s, 1)
    base = engine.Model(s, base_w)
    seq = np.concatenate([r["prompts"][n // wl.group], r["toks"][n][:T]]).astype(np.int32)
    lp, kl, kl_rev = engine.teacher_forced_kl(r["model"], base, r["kv"], dev_i32(seq[None, :]), P)
    lp, kl, kl_rev = lp.cpu().numpy()[0], kl.cpu().numpy()[0], kl_rev.cpu().numpy()[0]
    np.testing.assert_array_equal(lp.view(np.uint32), r["lps"][n, :T].view(np.uint32))
    ts = np.array([0, 1, 17, T - 1])
    sd = shape_dict(s)
    la = om.forward(sd, r["weights"], seq[:P + ts.max()], positions=P - 1 + ts)
    lb = om.forward(sd, base_w, seq[:P + ts.max()], positions=P - 1 + ts)
    want, want_rev = opol.kl_rows(la, lb)
    sens, sens_rev = kl_sensitivity(la, lb)
    tol = 2 * LOGIT_TOL * sens + 4 * LOGIT_TOL ** 2
    tol_rev = 2 * LOGIT_TOL * sens_rev + 4 * LOGIT_TOL ** 2
    assert np.all(np.abs(kl[ts] - want) <= tol), (kl[ts], want, tol)
    assert np.all(np.abs(kl_rev[ts] - want_rev) <= tol_rev), (kl_rev[ts], want_rev, tol_rev)
    assert np.all(kl > 0) and np.all(np.isfinite(kl))
