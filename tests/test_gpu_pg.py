"""GPU parity of the teacher-forced log-probs (dash_teacher_forced_logprobs) and the
policy-gradient loss (dash_pg_loss) against the oracle, and their consistency with
the log-probs the rollout recorded while sampling."""
import numpy as np
import pytest
import torch

from oracle import advantage as oa
from oracle import pg as opg
from paper_2505_17218_amd import _lib as L
from paper_2505_17218_amd import engine, synth

from gpu_util import dev_i32, make_kv, require_gpu, shape_dict

pytestmark = pytest.mark.gpu

BF16_A = synth.Shape("bf16-hd64", 2, 256, 8, 2, 64, 512, 1000, 1e6, synth.DT_BF16)
BF16_B = synth.Shape("bf16-hd128", 2, 384, 6, 2, 128, 768, 2051, 1e6, synth.DT_BF16)
# log-prob tolerance: a log-softmax value moves by at most twice the logits' error
LP_TOL = {synth.DT_F32: 2e-4, synth.DT_BF16: 6e-2}


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def _seqs(shape, n, P, T, seed):
    wl = synth.Workload("t", shape, n, 1, P, T)
    prompts = synth.make_prompts(wl, seed)
    comp = np.random.default_rng(seed).integers(0, shape.vocab, (n, T)).astype(np.int32)
    return prompts, comp, np.concatenate([prompts, comp], axis=1).astype(np.int32)


@pytest.mark.parametrize("shape,n,P,T", [(synth.TINY, 5, 16, 20), (BF16_A, 3, 40, 33), (BF16_B, 2, 64, 70)])
def test_teacher_forced_logprobs_match_oracle(shape, n, P, T):
    w = synth.make_weights(shape, 11)
    prompts, comp, seqs = _seqs(shape, n, P, T, 11)
    model = engine.Model(shape, w)
    kv = make_kv(model, 32 if shape.dtype == synth.DT_BF16 else 16, n, P + T)
    lp = engine.teacher_forced_logprobs(model, kv, dev_i32(seqs), P).cpu().numpy()
    sd = shape_dict(shape)
    worst = 0.0
    for b in range(n):
        want = opg.teacher_forced_logprobs(sd, w, prompts[b], comp[b])
        worst = max(worst, float(np.abs(want - lp[b]).max()))
    assert worst <= LP_TOL[shape.dtype], worst
    assert kv.free_pages == kv.pool.numel() // L.dash_kv_page_bytes(model.handle, kv.page_size)


def test_teacher_forced_chunking_is_bit_identical():
    """One sequence per chunk or several: the same bits (the kernels are batch-invariant)."""
    shape = BF16_A
    w = synth.make_weights(shape, 12)
    _, _, seqs = _seqs(shape, 5, 33, 20, 12)
    model = engine.Model(shape, w)
    kv = make_kv(model, 32, 5, 53)
    a = engine.teacher_forced_logprobs(model, kv, dev_i32(seqs), 33, seqs_per_chunk=1).cpu().numpy()
    b = engine.teacher_forced_logprobs(model, kv, dev_i32(seqs), 33, seqs_per_chunk=3).cpu().numpy()
    np.testing.assert_array_equal(a, b)


@pytest.mark.parametrize("shape", [synth.TINY, BF16_B])
def test_recompute_matches_rollout_logprobs(shape):
    """The teacher-forced recompute of the rollout's own tokens reproduces the log-probs
    recorded while sampling (temperature 1) bit for bit: every context here fits one
    decode-attention split, the prefill and decode attention run the same per-column
    block step, the GEMMs and norms are batch-invariant, and the log-normaliser is
    summed in the sampler's order.  Then the PG loss over the kept samples matches the
    oracle formula on the recomputed log-probs."""
    n_prompts, G, P, T = 3, 4, 24, 30
    w = synth.make_weights(shape, 13)
    wl = synth.Workload("t", shape, n_prompts, G, P, T)
    prompts = synth.make_prompts(wl, 13)
    model = engine.Model(shape, w)
    ps = 32 if shape.dtype == synth.DT_BF16 else 16
    N = n_prompts * G
    kv = make_kv(model, ps, N, P + T)
    ro = engine.Rollout(model, kv, n_prompts, P, G, T)
    toks, lps = ro.run(dev_i32(prompts), 1.0, 5, use_graph=False)
    toks = toks.cpu().numpy().copy()
    lps = lps.cpu().numpy().copy()
    seqs = np.concatenate([np.repeat(prompts, G, axis=0), toks], axis=1).astype(np.int32)
    assert P + T <= kv.split_keys
    rec = engine.teacher_forced_logprobs(model, kv, dev_i32(seqs), P).cpu().numpy()
    np.testing.assert_array_equal(rec.view(np.uint32), lps.view(np.uint32))
    rewards = synth.make_rewards(n_prompts, G, "beta0.5", 13)
    adv, kept = engine.advantage_filter(torch.from_numpy(rewards).cuda(), G, L.DASH_ADV_STD_SAMPLE, 1e-6, 0.1)
    lengths = np.random.default_rng(0).integers(1, T + 1, N).astype(np.int32)
    loss, seq = engine.pg_loss(torch.from_numpy(rec).cuda(), adv, kept, dev_i32(lengths))
    want_loss, want_seq = opg.pg_loss(rec, adv.cpu().numpy(), kept.cpu().numpy(), lengths)
    assert abs(float(loss.item()) - want_loss) <= 1e-12 * max(1.0, abs(want_loss))
    k = kept.cpu().numpy()
    np.testing.assert_allclose(seq.cpu().numpy()[k], want_seq[k], rtol=1e-12, atol=1e-12)


def test_pg_loss_edge_cases():
    lp = torch.tensor([[-1.0, -2.0], [-0.5, -0.5], [-3.0, 0.0]], device="cuda")
    adv = torch.tensor([1.0, -2.0, 0.5], device="cuda")
    loss, _ = engine.pg_loss(lp, adv, dev_i32([0, 1]))
    assert abs(float(loss.item()) - 1.0 / 3.0) < 1e-15
    loss, _ = engine.pg_loss(lp, adv, dev_i32([]))  # nothing kept
    assert float(loss.item()) == 0.0
