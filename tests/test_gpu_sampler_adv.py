"""GPU parity of dash_sample, dash_group_advantage_filter and dash_live_compact
against the oracle (tokens, advantages and index sets bit-exact)."""
import numpy as np
import pytest
import torch

from oracle import advantage as oa
from oracle import rollout as oro
from oracle import sampler as osm
from paper_2505_17218_amd import _lib as L
from paper_2505_17218_amd import engine, synth

from gpu_util import dev_i32, require_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


# log-probability tolerance: fp32 online log-sum-exp over up to 151936 terms
# (relative error of the sum ~1e-6) against the float64 oracle
LP_ATOL, LP_RTOL = 5e-5, 2e-6


@pytest.mark.parametrize("rows,vocab,temp,seed,scale", [
    (16, 512, 1.0, 2, 1.0), (64, 151936, 1.0, 2, 2.0), (33, 151936, 0.7, 12345, 1.0),
    (7, 5, 1.0, 3, 1.0), (5, 1, 1.0, 4, 1.0), (9, 1001, 2.5, 0xFFFFFFFFFFFF, 3.0), (1024, 4096, 1.0, 2, 1.0)])
def test_sample_bitexact(rows, vocab, temp, seed, scale):
    logits = synth.make_logits(rows, vocab, seed=rows + vocab, scale=scale)
    rng = np.random.default_rng(vocab)
    uid = rng.integers(0, 1 << 20, rows).astype(np.int32)
    step = rng.integers(0, 2048, rows).astype(np.int32)
    toks, lps = engine.sample(torch.from_numpy(logits).cuda(), dev_i32(uid), dev_i32(step), temp, seed)
    want_t, want_lp = osm.sample(logits, uid, step, temp, seed)
    np.testing.assert_array_equal(toks.cpu().numpy(), want_t)
    np.testing.assert_allclose(lps.cpu().numpy(), want_lp, atol=LP_ATOL, rtol=LP_RTOL)


def test_sampler_screening_bound_exhaustive():
    """The cheap noise that screens vocab entries stays within the sampler's tolerance
    of the exact noise for every one of the 2^23 values u can take (on this GPU)."""
    err, tol = L.dash_sampler_check()
    assert 0.0 < err and 4.0 * err <= tol, (err, tol)


def test_bf16_rounding_instruction_exhaustive():
    """The GPU's float32 -> bfloat16 conversion, which every bf16 store of the kernels
    uses, agrees with integer round-to-nearest-even of the bit pattern on all 2^32
    inputs (NaNs included), on this device."""
    assert L.dash_bf16_round_check() == 0


@pytest.mark.parametrize("case", ["flat", "large", "near_ties", "cold", "two_level"])
def test_sample_screening_adversarial(case):
    """Rows built so that many entries land close to the best score: flat logits (the
    noise alone decides), large magnitudes (wide fp32 rounding), near-ties spaced below
    the screening margin, a cold temperature, and a few dominant entries."""
    rows, V = 64, 151936
    rng = np.random.default_rng(["flat", "large", "near_ties", "cold", "two_level"].index(case))
    temp = 1.0
    if case == "flat":
        logits = np.zeros((rows, V), np.float32)
    elif case == "large":
        logits = (3e4 + rng.standard_normal((rows, V))).astype(np.float32)
    elif case == "near_ties":
        logits = (rng.integers(0, 64, (rows, V)) * np.float32(2e-6)).astype(np.float32)
    elif case == "cold":
        logits = rng.standard_normal((rows, V)).astype(np.float32) * np.float32(0.01)
        temp = 0.003
    else:
        logits = np.full((rows, V), -5.0, np.float32)
        logits[:, rng.integers(0, V, 6)] = 8.0
    uid = np.arange(rows, dtype=np.int32)
    step = np.full(rows, 17, np.int32)
    toks, _ = engine.sample(torch.from_numpy(logits).cuda(), dev_i32(uid), dev_i32(step), temp, 31)
    want_t, _ = osm.sample(logits, uid, step, temp, 31)
    np.testing.assert_array_equal(toks.cpu().numpy(), want_t)


def test_sample_row_of_stride_and_nonfinite():
    V, R = 1000, 6
    wide = synth.make_logits(R, V + 24, seed=9)  # row stride 1024 > vocab
    wide[1, 17] = np.inf
    wide[2, :V] = np.nan   # no finite logit: token -1
    wide[3, 5] = np.nan
    wide[4, 100:300] = -np.inf
    dl = torch.from_numpy(wide).cuda()[:, :V]
    row_of = np.array([0, 1, 3, 4, 5, 0, 1, 4], np.int32)
    B = row_of.size
    uid = np.arange(B, dtype=np.int32) * 7
    step = np.full(B, 3, np.int32)
    toks, lps = engine.sample(dl, dev_i32(uid), dev_i32(step), 1.0, 99, row_of=dev_i32(row_of))
    want_t, want_lp = osm.sample(wide[:, :V], uid, step, 1.0, 99, row_of=row_of)
    np.testing.assert_array_equal(toks.cpu().numpy(), want_t)
    np.testing.assert_allclose(lps.cpu().numpy(), want_lp, atol=LP_ATOL, rtol=LP_RTOL)
    toks2, _ = engine.sample(dl, dev_i32([0]), dev_i32([0]), 1.0, 1, row_of=dev_i32([2]))
    assert int(toks2.item()) == -1


@pytest.mark.parametrize("V,ld,off", [(1000, 1003, 0), (4096, 4096, 1), (1001, 1004, 0), (151936, 151937, 0)])
def test_sample_row_layouts(V, ld, off):
    """Rows the sampler cannot read in 16-byte groups (a row stride or start that is not a
    multiple of four floats, a vocabulary that is not) draw the same tokens as the oracle,
    and as the same logits in an aligned copy (the two load paths agree)."""
    R = 9
    buf = synth.make_logits(R * ld + off + 4, 1, seed=V + ld).reshape(-1)
    view = buf[off:off + R * ld].reshape(R, ld)[:, :V]
    uid = np.arange(R, dtype=np.int32) * 13
    step = np.full(R, 5, np.int32)
    d = torch.from_numpy(buf).cuda()[off:off + R * ld].view(R, ld)[:, :V]
    toks, lps = engine.sample(d, dev_i32(uid), dev_i32(step), 1.0, 77)
    want_t, want_lp = osm.sample(np.ascontiguousarray(view), uid, step, 1.0, 77)
    np.testing.assert_array_equal(toks.cpu().numpy(), want_t)
    np.testing.assert_allclose(lps.cpu().numpy(), want_lp, atol=LP_ATOL, rtol=LP_RTOL)
    t2, lp2 = engine.sample(torch.from_numpy(np.ascontiguousarray(view)).cuda(), dev_i32(uid), dev_i32(step), 1.0, 77)
    np.testing.assert_array_equal(t2.cpu().numpy(), toks.cpu().numpy())
    np.testing.assert_array_equal(lp2.cpu().numpy().view(np.uint32), lps.cpu().numpy().view(np.uint32))


def test_sample_deterministic_and_independent_of_batch_position():
    logits = synth.make_logits(8, 151936, seed=5)
    uid = np.arange(8, dtype=np.int32)
    step = np.full(8, 10, np.int32)
    a, _ = engine.sample(torch.from_numpy(logits).cuda(), dev_i32(uid), dev_i32(step), 1.0, 7)
    perm = np.array([3, 1, 7, 0, 2, 6, 5, 4])
    b, _ = engine.sample(torch.from_numpy(logits[perm]).cuda(), dev_i32(uid[perm]), dev_i32(step), 1.0, 7)
    np.testing.assert_array_equal(a.cpu().numpy()[perm], b.cpu().numpy())


@pytest.mark.parametrize("G", [1, 2, 3, 4, 5, 8, 16, 33, 64, 100, 1024, 1500, 4096, 65536])
@pytest.mark.parametrize("mode", [L.DASH_ADV_MEAN_ONLY, L.DASH_ADV_STD_POP, L.DASH_ADV_STD_SAMPLE, L.DASH_ADV_LOO])
def test_advantage_filter_bitexact(G, mode):
    """Every mode and group size, from wave-sized groups to one group of 65536 (the
    single-path baseline of Eq. (3) over a whole batch), bit-exact against the oracle."""
    n_groups = max(1, 4096 // G)
    if mode == L.DASH_ADV_LOO and G == 1:  # the leave-one-out baseline needs two samples per group
        r = torch.zeros(n_groups, dtype=torch.float32, device="cuda")
        with pytest.raises(L.DashError) as e:
            engine.advantage_filter(r, 1, mode, 1e-6, 0.1)
        assert e.value.status == L.DASH_EINVAL
        return
    r = synth.make_rewards(n_groups, G, "beta0.5", seed=G)
    # mix in continuous rewards so |A| lands everywhere, including near tau
    cont = np.random.default_rng(G).standard_normal(r.size).astype(np.float32) * np.float32(0.3)
    for rr in (r, (r + cont).astype(np.float32)):
        adv, kept = engine.advantage_filter(torch.from_numpy(rr).cuda(), G, mode, 1e-6, 0.1)
        want = oa.group_advantage(rr, G, mode, 1e-6)
        np.testing.assert_array_equal(adv.cpu().numpy().view(np.uint32), want.view(np.uint32))
        np.testing.assert_array_equal(kept.cpu().numpy(), oa.gradient_filter(want, 0.1))


@pytest.mark.parametrize("n_groups,G", [(4, 4), (128, 8), (512, 8), (8192, 8)])
def test_advantage_workload_sizes(n_groups, G):
    kind = "bernoulli0.5" if G == 4 else "beta0.5"
    r = synth.make_rewards(n_groups, G, kind, seed=0)
    adv, kept = engine.advantage_filter(torch.from_numpy(r).cuda(), G, L.DASH_ADV_STD_SAMPLE, 1e-6, 0.1)
    want = oa.group_advantage(r, G, oa.STD_SAMPLE, 1e-6)
    np.testing.assert_array_equal(adv.cpu().numpy().view(np.uint32), want.view(np.uint32))
    np.testing.assert_array_equal(kept.cpu().numpy(), oa.gradient_filter(want, 0.1))


def test_advantage_tau_zero_and_tiny():
    r = synth.make_rewards(64, 8, "beta0.5", seed=1)
    d = torch.from_numpy(r).cuda()
    _, kept0 = engine.advantage_filter(d, 8, L.DASH_ADV_MEAN_ONLY, 1e-6, 0.0)
    assert kept0.numel() == r.size
    _, kept1 = engine.advantage_filter(d, 8, L.DASH_ADV_MEAN_ONLY, 1e-6, float(np.finfo(np.float32).smallest_subnormal))
    want = oa.gradient_filter(oa.group_advantage(r, 8, oa.MEAN_ONLY), np.finfo(np.float32).smallest_subnormal)
    np.testing.assert_array_equal(kept1.cpu().numpy(), want)


@pytest.mark.parametrize("n,eos", [(0, -1), (1, -1), (1000, -1), (4096, 7), (3000, -1), (9000, 3)])
def test_live_compact_matches_oracle(n, eos):
    """dash_live_compact against the oracle's row bookkeeping (oracle.rollout.live_compact),
    bit for bit: which rows go on, their order, and their advanced positions and steps."""
    rng = np.random.default_rng(n + 1)
    uid = rng.permutation(16384)[:n].astype(np.int32)
    budget = rng.integers(1, 50, 16384).astype(np.int32)
    step = rng.integers(0, 50, n).astype(np.int32)
    tok = rng.integers(0, 16, n).astype(np.int32)
    slot = rng.integers(0, 1 << 16, n).astype(np.int32)
    pos = rng.integers(0, 4096, n).astype(np.int32)
    m = max(n, 1)
    outs = [torch.full((m,), -7, dtype=torch.int32, device="cuda") for _ in range(5)]
    cnt = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    ins = [dev_i32(a if n else np.zeros(1)) for a in (tok, slot, pos, step, uid)]
    L.dash_live_compact(*[t.data_ptr() for t in ins], dev_i32(budget).data_ptr(), eos, n,
                        *[t.data_ptr() for t in outs], cnt.data_ptr(), engine.stream_handle())
    want = oro.live_compact(tok, slot, pos, step, uid, budget, eos)
    k = int(cnt.item())
    assert k == len(want[0])
    for g, w in zip(outs, want):
        np.testing.assert_array_equal(g.cpu().numpy()[:k], w)
        assert (g.cpu().numpy()[k:] == -7).all()  # nothing written past the live rows


def test_sample_status_bit_and_row_max_lse():
    """A row with no finite logit draws -1 and sets DASH_ST_NO_FINITE_LOGIT in the status word;
    non-finite entries are never drawn; the per-row (max, log normaliser) output matches the
    float64 values of softmax(l / T), and the drawn token's log-prob equals l / T minus it."""
    rows, V, temp, seed = 6, 1000, 0.8, 9
    lg = synth.make_logits(rows, V, seed=5, scale=2.0)
    lg[1, :] = np.nan                 # nothing finite
    lg[2, :] = -np.inf
    lg[2, 17] = 0.5                   # one finite entry
    lg[3, 5] = np.inf                 # never drawn
    lg[4, :] = -np.inf                # nothing finite
    d = torch.from_numpy(lg).cuda()
    ml = torch.full((rows, 2), 7.0, dtype=torch.float32, device="cuda")
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    uid, step = dev_i32(np.arange(rows)), dev_i32(np.zeros(rows))
    toks, lps = engine.sample(d, uid, step, temp, seed, row_max_lse=ml, status=st)
    want, want_lp = osm.sample(lg, np.arange(rows), np.zeros(rows), temp, seed)
    toks = toks.cpu().numpy()
    np.testing.assert_array_equal(toks, want)
    assert want[1] == -1 and want[4] == -1 and want[2] == 17 and want[3] != 5
    assert int(st.item()) == L.DASH_ST_NO_FINITE_LOGIT
    ml, lps = ml.cpu().numpy(), lps.cpu().numpy()
    T32 = np.float32(temp)
    for r in (0, 2, 3, 5):
        z = (lg[r][np.isfinite(lg[r])] / T32).astype(np.float64)
        m = z.max()
        lse = m + np.log(np.exp(z - m).sum())
        assert ml[r, 0] == np.float32(m)
        assert abs(ml[r, 1] - lse) <= LP_ATOL + LP_RTOL * abs(lse)
        assert abs(lps[r] - (np.float32(lg[r, toks[r]] / T32) - ml[r, 1])) <= 1e-5
    assert np.isnan(ml[[1, 4]]).all() and np.isnan(lps[[1, 4]]).all()
    # rows with finite logits only: the bit stays clear; no status pointer is fine too
    st.zero_()
    engine.sample(d[[0, 2, 3, 5]].contiguous(), dev_i32(np.arange(4)), dev_i32(np.zeros(4)), temp, seed, status=st)
    engine.sample(d, uid, step, temp, seed)
    torch.cuda.synchronize()
    assert int(st.item()) == 0
