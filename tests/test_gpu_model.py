"""GPU parity of dash_prefill / dash_decode_step / dash_rollout against the oracle.

For every generated position the GPU's logits are compared with the oracle's
teacher-forced logits for the same tokens (max abs diff <= 1e-4 for float32
shapes, <= 3e-2 for bfloat16 shapes), and the oracle sampler applied to the
GPU's logits must reproduce the GPU's tokens bit for bit."""
import numpy as np
import pytest
import torch

from oracle import model as om
from oracle import sampler as osm
from paper_2505_17218_amd import _lib as L
from paper_2505_17218_amd import engine, synth

from gpu_util import dev_i32, make_kv, require_gpu, run_stepwise, shape_dict

pytestmark = pytest.mark.gpu

TOL = {synth.DT_F32: 1e-4, synth.DT_BF16: 3e-2}


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


# bf16 shapes small enough for the oracle, covering both head dims, GQA groups
# of 3/4/7, vocab tails (not a multiple of 128) and partial prompt pages.
BF16_A = synth.Shape("bf16-hd64", 2, 256, 8, 2, 64, 512, 1000, 1e6, synth.DT_BF16)
BF16_B = synth.Shape("bf16-hd128", 2, 384, 6, 2, 128, 768, 2051, 1e6, synth.DT_BF16)
BF16_C = synth.Shape("bf16-gqa7", 1, 448, 7, 1, 64, 320, 700, 1e4, synth.DT_BF16)


def _check_run(shape, w, prompts, G, T, run: "object", temp, seed, tol):
    sd = shape_dict(shape)
    N = prompts.shape[0] * G
    worst = 0.0
    for n in range(N):
        ref = om.rollout_logits(sd, w, prompts[n // G], run.tokens[n])
        err = np.abs(ref - run.logits[:, n, :]).max()
        worst = max(worst, err)
    assert worst <= tol, f"max |logits - oracle| = {worst}"
    # the oracle sampler on the GPU's logits reproduces the GPU's tokens
    for t in range(T):
        want, want_lp = osm.sample(run.logits[t], np.arange(N), np.full(N, t), temp, seed)
        np.testing.assert_array_equal(run.tokens[:, t], want)
        np.testing.assert_allclose(run.logprobs[:, t], want_lp, atol=5e-5, rtol=2e-6)
    return worst


@pytest.mark.parametrize("page_size", [16, 7, 64])
def test_tiny_fp32_stepwise_matches_oracle(page_size):
    wl = synth.WORKLOADS["tiny"]
    shape = wl.shape
    w = synth.make_weights(shape, 0)
    prompts = synth.make_prompts(wl, 0)
    model = engine.Model(shape, w)
    kv = make_kv(model, page_size, wl.n_seqs, wl.prompt_len + wl.gen_len)
    run = run_stepwise(model, kv, prompts, wl.group, wl.gen_len, wl.temperature, synth.sampler_seed(0))
    worst = _check_run(shape, w, prompts, wl.group, wl.gen_len, run, wl.temperature, synth.sampler_seed(0),
                       TOL[shape.dtype])
    print(f"tiny fp32 ps={page_size}: max |dlogits| = {worst:.3g}")


@pytest.mark.parametrize("shape,n_prompts,G,P,T", [
    (BF16_A, 3, 4, 40, 40), (BF16_B, 2, 4, 64, 33), (BF16_C, 2, 2, 31, 20), (BF16_A, 1, 2, 600, 6)])
def test_bf16_stepwise_matches_oracle(shape, n_prompts, G, P, T):
    w = synth.make_weights(shape, 1)
    wl = synth.Workload("t", shape, n_prompts, G, P, T)
    prompts = synth.make_prompts(wl, 1)
    model = engine.Model(shape, w)
    kv = make_kv(model, 32, n_prompts * G, P + T)
    run = run_stepwise(model, kv, prompts, G, T, 1.0, 77)
    worst = _check_run(shape, w, prompts, G, T, run, 1.0, 77, TOL[shape.dtype])
    print(f"{shape.name} P={P} T={T}: max |dlogits| = {worst:.3g}")


@pytest.mark.parametrize("max_seqs,split", [(4, 128), (1024, 512), (2048, 1024)])
def test_bf16_split_length_follows_capacity(max_seqs, split):
    """The decode-attention split length is fixed per cache from its capacity (head dim 64:
    three waves per SIMD): a small cache cuts a 600-key context into 128-key splits merged
    by the combine kernel, a larger one into two 512-key splits, a large one reads it as a
    single 1024-key split.  All match the oracle."""
    shape = BF16_A
    w = synth.make_weights(shape, 1)
    wl = synth.Workload("t", shape, 2, 2, 600, 6)
    prompts = synth.make_prompts(wl, 1)
    model = engine.Model(shape, w)
    kv = engine.KVCache(model, 32, max_seqs, 606, 4 * 19 + 8)  # pages for the 4 rows used
    assert kv.split_keys == split
    run = run_stepwise(model, kv, prompts, 2, 6, 1.0, 77)
    worst = _check_run(shape, w, prompts, 2, 6, run, 1.0, 77, TOL[shape.dtype])
    print(f"split {split}: max |dlogits| = {worst:.3g}")


@pytest.mark.parametrize("P,n_splits", [(1800, 15), (2600, 21)])
def test_bf16_many_attention_splits(P, n_splits):
    """A small cache keeps 128-key splits, so long contexts are merged from many splits:
    15 (the merge with every load issued up front, up to 16 splits) and 21 (the merge
    that loads split by split).  Both match the oracle."""
    shape = BF16_A
    w = synth.make_weights(shape, 1)
    T = 3
    wl = synth.Workload("t", shape, 1, 2, P, T)
    prompts = synth.make_prompts(wl, 1)
    model = engine.Model(shape, w)
    kv = engine.KVCache(model, 32, 4, P + T, 2 * ((P + T + 31) // 32) + 8)
    assert kv.split_keys == 128 and -(-(P + T) // 128) == n_splits
    run = run_stepwise(model, kv, prompts, 2, T, 1.0, 77)
    worst = _check_run(shape, w, prompts, 2, T, run, 1.0, 77, TOL[shape.dtype])
    print(f"P={P} ({n_splits} splits): max |dlogits| = {worst:.3g}")


def test_prefill_in_chunks_is_bit_identical():
    """A workspace for 5 prompts makes dash_prefill take 8 prompts in two equal chunks of 4;
    the logits, and a decode step over the cache it wrote, match a one-chunk prefill bit for bit."""
    shape, G, P = BF16_A, 2, 40
    w = synth.make_weights(shape, 12)
    prompts = synth.make_prompts(synth.Workload("t", shape, 8, G, P, 2), 12)
    model = engine.Model(shape, w)
    slots = list(range(8 * G))
    outs = []
    for ws in (None, model.workspace(5 * P, 0)):
        kv = make_kv(model, 32, 8 * G, P + 1)
        logits = engine.prefill(model, kv, dev_i32(prompts), G, slots, ws=ws).cpu().numpy()
        L.dash_kv_reserve(kv.handle, slots, P + 1, engine.stream_handle())
        tok = dev_i32(np.arange(8 * G) % shape.vocab)
        step = engine.decode_step(model, kv, tok, dev_i32(np.arange(8 * G)), dev_i32(np.full(8 * G, P)))
        outs.append((logits, step.cpu().numpy()))
    np.testing.assert_array_equal(outs[0][0], outs[1][0])
    np.testing.assert_array_equal(outs[0][1], outs[1][1])


def test_bf16_large_batch_gemm_tiles():
    """160 decode rows (M > 128 with a tail) through the MFMA GEMMs; checked on sampled rows."""
    shape = BF16_A
    w = synth.make_weights(shape, 2)
    wl = synth.Workload("t", shape, 40, 4, 20, 4)
    prompts = synth.make_prompts(wl, 2)
    model = engine.Model(shape, w)
    kv = make_kv(model, 32, 160, 24)
    run = run_stepwise(model, kv, prompts, 4, 4, 1.0, 5)
    sd = shape_dict(shape)
    for n in (0, 1, 63, 64, 127, 128, 129, 159):
        ref = om.rollout_logits(sd, w, prompts[n // 4], run.tokens[n])
        assert np.abs(ref - run.logits[:, n, :]).max() <= TOL[shape.dtype]


# a long down-projection reduction (d_ff = 4096 >= 4096): split-K on the narrow small-batch tiles
BF16_D = synth.Shape("bf16-ff4096", 1, 256, 4, 2, 64, 4096, 500, 1e6, synth.DT_BF16)


@pytest.mark.parametrize("n_prompts", [10, 75, 150])
def test_bf16_gemm_tile_regimes(n_prompts):
    """Decode batches of 40, 300 and 600 rows select different GEMM tiles (narrow
    small-batch tiles, 64x64, 128x256 for the split-K down projection); all match the
    oracle, and a row's logits do not depend on the regime its batch falls in."""
    shape = BF16_D
    w = synth.make_weights(shape, 8)
    wl = synth.Workload("t", shape, 150, 4, 12, 3)
    prompts = synth.make_prompts(wl, 8)[:n_prompts]
    model = engine.Model(shape, w)
    kv = make_kv(model, 32, n_prompts * 4, 15)
    run = run_stepwise(model, kv, prompts, 4, 3, 1.0, 5)
    sd = shape_dict(shape)
    for n in sorted({0, 3, n_prompts * 2 + 1, n_prompts * 4 - 1}):
        ref = om.rollout_logits(sd, w, prompts[n // 4], run.tokens[n])
        assert np.abs(ref - run.logits[:, n, :]).max() <= TOL[shape.dtype], n
    if n_prompts != 10:  # rows of the first 10 prompts: same logits as in the 40-row batch
        small = run_stepwise(model, make_kv(model, 32, 40, 15), prompts[:10], 4, 3, 1.0, 5)
        np.testing.assert_array_equal(small.logits[0], run.logits[0][:40])


# d_ff = 2240 (18 columns of 128-wide SwiGLU tile pairs): a 1024-row decode batch runs
# gate/up on 128x256 tiles (144, under one round), a 40-row batch on 64x64 tiles
BF16_E = synth.Shape("bf16-ff2240", 1, 256, 4, 2, 64, 2240, 500, 1e6, synth.DT_BF16)


def test_bf16_swiglu_tile_regimes_bitexact():
    """1024 decode rows (128x256 SwiGLU tiles) give every row the same logits, bit for bit,
    as a 40-row batch (64x64 tiles), and match the oracle."""
    shape = BF16_E
    w = synth.make_weights(shape, 9)
    wl = synth.Workload("t", shape, 256, 4, 10, 2)
    prompts = synth.make_prompts(wl, 9)
    model = engine.Model(shape, w)
    big = run_stepwise(model, make_kv(model, 32, 1024, 12), prompts, 4, 2, 1.0, 5)
    small = run_stepwise(model, make_kv(model, 32, 40, 12), prompts[:10], 4, 2, 1.0, 5)
    np.testing.assert_array_equal(small.logits[1], big.logits[1][:40])  # the decode step (M = 1024 vs 40)
    sd = shape_dict(shape)
    for n in (0, 511, 1023):
        ref = om.rollout_logits(sd, w, prompts[n // 4], big.tokens[n])
        assert np.abs(ref - big.logits[:, n, :]).max() <= TOL[shape.dtype], n


# d_ff = 8320 (65 columns of 128-wide SwiGLU tile pairs): at 1024 rows one round of 256x256
# tiles covers 8192 columns (260 tiles would leave a last round of 4), so gate/up runs as two
# launches, 256x256 over those columns and 64x128 over the last 128; 40 rows on 64x64 tiles
BF16_I = synth.Shape("bf16-ff8320", 1, 256, 4, 2, 64, 8320, 500, 1e6, synth.DT_BF16)


def test_bf16_swiglu_tile_rounds_bitexact():
    """The 1024-row gate/up tiling chosen by how the tiles fill the GPU (one round of
    256x256 tiles, the remaining columns on 64x128 tiles) gives the rows it shares with a
    40-row batch the same logits, bit for bit, and matches the oracle."""
    shape = BF16_I
    w = synth.make_weights(shape, 12)
    wl = synth.Workload("t", shape, 256, 4, 10, 2)
    prompts = synth.make_prompts(wl, 12)
    model = engine.Model(shape, w)
    big = run_stepwise(model, make_kv(model, 32, 1024, 12), prompts, 4, 2, 1.0, 5)
    small = run_stepwise(model, make_kv(model, 32, 40, 12), prompts[:10], 4, 2, 1.0, 5)
    np.testing.assert_array_equal(small.logits[1], big.logits[1][:40])  # the decode step (M = 1024 vs 40)
    sd = shape_dict(shape)
    for n in (0, 517, 1023):
        ref = om.rollout_logits(sd, w, prompts[n // 4], big.tokens[n])
        assert np.abs(ref - big.logits[:, n, :]).max() <= TOL[shape.dtype], n


# d_ff = 8192 (128 SwiGLU tiles of 64 column pairs): gate/up runs on 64x128 tiles with three
# k-steps in flight up to 64 rows, on 64x64 tiles at 65-128 rows, on 64x128 tiles with two
# k-steps in flight at 129-256 rows, on 128x128 tiles at 300 rows, on 256x256 tiles at 480
# and 1024 rows (one round of 128 / 256 of them) and on 128x128 tiles again at 2048 rows
# (512 = two exact rounds of 256x256, 1024 = four of 128x256); the down projection
# (K = 8192, split) on 64x32 tiles four k-steps ahead, 64x64 tiles three or two k-steps
# ahead, direct-to-LDS 128x128 tiles (480 rows), 128x256 or 256x256; the output projection
# on 64x32 tiles, 64x64 tiles three or two k-steps ahead, direct-to-LDS or 256x256 tiles
BF16_G = synth.Shape("bf16-ff8192", 1, 256, 4, 2, 64, 8192, 500, 1e6, synth.DT_BF16)


def test_bf16_gemm_regimes_across_batch_sizes_bitexact():
    """Batches of 10 to 512 prompts (prefill 100 to 5120 rows, decode 40 to 2048 rows) run
    every gate/up, down and output projection tiling; the rows they share get the same
    logits bit for bit, and sampled rows match the oracle."""
    shape = BF16_G
    w = synth.make_weights(shape, 11)
    wl = synth.Workload("t", shape, 512, 4, 10, 2)
    prompts = synth.make_prompts(wl, 11)
    model = engine.Model(shape, w)
    runs = {n: run_stepwise(model, make_kv(model, 32, 4 * n, 12), prompts[:n], 4, 2, 1.0, 5)
            for n in (10, 25, 50, 75, 120, 256, 512)}
    for n in (25, 50, 75, 120, 256, 512):
        np.testing.assert_array_equal(runs[10].logits[0], runs[n].logits[0][:40])  # prefill
        np.testing.assert_array_equal(runs[10].logits[1], runs[n].logits[1][:40])  # decode step
    sd = shape_dict(shape)
    for n_prompts, n in ((10, 0), (25, 99), (50, 199), (75, 299), (120, 479), (256, 1023), (512, 2047)):
        run = runs[n_prompts]
        ref = om.rollout_logits(sd, w, prompts[n // 4], run.tokens[n])
        assert np.abs(ref - run.logits[:, n, :]).max() <= TOL[shape.dtype], (n_prompts, n)


@pytest.mark.parametrize("ff,n_prompts,rest", [(8960, 256, "64x128"), (8960, 512, "128x128"),
                                              (11008, 256, "128x256"), (4864, 512, "128x128"),
                                              (8960, 275, "128x256")])
def test_bf16_swiglu_column_split_bitexact(ff, n_prompts, rest):
    """Gate/up widths of the 0.5B, 1.5B and 3B shapes at 1024 and 2048 rows, where whole
    rounds of 256x256 tiles would leave a last round under half full: the columns of the
    whole rounds run as one launch and the rest (on the tile named by `rest`) as another
    (1100 rows, 275 prompts: partial row tiles in both launches, columns split at 6528).
    The rows shared with a 40-row batch (64x64 tiles) get the same logits bit for bit, and
    sampled rows match the oracle."""
    shape = synth.Shape(f"bf16-ff{ff}", 1, 256, 4, 2, 64, ff, 500, 1e6, synth.DT_BF16)
    w = synth.make_weights(shape, 13)
    wl = synth.Workload("t", shape, n_prompts, 4, 10, 2)
    prompts = synth.make_prompts(wl, 13)
    model = engine.Model(shape, w)
    N = 4 * n_prompts
    big = run_stepwise(model, make_kv(model, 32, N, 12), prompts, 4, 2, 1.0, 5)
    small = run_stepwise(model, make_kv(model, 32, 40, 12), prompts[:10], 4, 2, 1.0, 5)
    np.testing.assert_array_equal(small.logits[1], big.logits[1][:40])  # the decode step (M = N vs 40)
    sd = shape_dict(shape)
    for n in (0, N // 2 + 1, N - 1):
        ref = om.rollout_logits(sd, w, prompts[n // 4], big.tokens[n])
        assert np.abs(ref - big.logits[:, n, :]).max() <= TOL[shape.dtype], n


# vocab 9000 (>= 8192 columns: the LM head's tiles): 64x256 up to 64 rows, 128x256 up to 128,
# 256x256 past that
BF16_H = synth.Shape("bf16-v9000", 1, 256, 4, 2, 64, 512, 9000, 1e6, synth.DT_BF16)


def test_bf16_lm_head_regimes_bitexact():
    """Batches of 10, 25 and 75 prompts put the LM head on 64x256, 128x256 and 256x256 tiles
    (prefill 10 / 25 / 75 rows, decode 40 / 100 / 300 rows); the rows they share get the same
    logits bit for bit, and sampled rows match the oracle."""
    shape = BF16_H
    w = synth.make_weights(shape, 14)
    prompts = synth.make_prompts(synth.Workload("t", shape, 75, 4, 10, 2), 14)
    model = engine.Model(shape, w)
    runs = {n: run_stepwise(model, make_kv(model, 32, 4 * n, 12), prompts[:n], 4, 2, 1.0, 5) for n in (10, 25, 75)}
    for n in (25, 75):
        np.testing.assert_array_equal(runs[10].logits[0], runs[n].logits[0][:40])  # prefill
        np.testing.assert_array_equal(runs[10].logits[1], runs[n].logits[1][:40])  # decode step
    sd = shape_dict(shape)
    for n_prompts, n in ((10, 0), (25, 99), (75, 299)):
        run = runs[n_prompts]
        ref = om.rollout_logits(sd, w, prompts[n // 4], run.tokens[n])
        assert np.abs(ref - run.logits[:, n, :]).max() <= TOL[shape.dtype], (n_prompts, n)


# q / k / v widths of 1536 / 256 / 256 (16 QKV tiles of 128 columns): a 1024-row batch runs the
# fused QKV kernel (bias, RoPE and the KV append in the GEMM epilogue), a 40-row batch the
# unfused GEMM and the standalone RoPE / append kernel
BF16_F = synth.Shape("bf16-qkv2048", 1, 256, 12, 2, 128, 512, 500, 1e6, synth.DT_BF16)


def test_bf16_fused_qkv_regimes_bitexact():
    """Fused and unfused QKV paths give the same rows the same logits, bit for bit, in the
    prefill (2560 vs 100 rows) and in a decode step (1024 vs 40 rows), and match the oracle."""
    shape = BF16_F
    w = synth.make_weights(shape, 10)
    wl = synth.Workload("t", shape, 256, 4, 10, 2)
    prompts = synth.make_prompts(wl, 10)
    model = engine.Model(shape, w)
    big = run_stepwise(model, make_kv(model, 32, 1024, 12), prompts, 4, 2, 1.0, 5)
    small = run_stepwise(model, make_kv(model, 32, 40, 12), prompts[:10], 4, 2, 1.0, 5)
    np.testing.assert_array_equal(small.logits[0], big.logits[0][:40])  # prefill
    np.testing.assert_array_equal(small.logits[1], big.logits[1][:40])  # decode step
    sd = shape_dict(shape)
    for n in (0, 777, 1023):
        ref = om.rollout_logits(sd, w, prompts[n // 4], big.tokens[n])
        assert np.abs(ref - big.logits[:, n, :]).max() <= TOL[shape.dtype], n


def test_page_size_and_batch_invariance_bf16():
    """Page size 32 vs 64 and a different batch composition give bit-identical tokens and logits."""
    shape = BF16_B
    w = synth.make_weights(shape, 3)
    wl = synth.Workload("t", shape, 3, 2, 45, 12)
    prompts = synth.make_prompts(wl, 3)
    model = engine.Model(shape, w)
    runs = []
    for ps in (32, 64):
        kv = make_kv(model, ps, 6, 64)
        runs.append(run_stepwise(model, kv, prompts, 2, 12, 1.0, 8))
    np.testing.assert_array_equal(runs[0].tokens, runs[1].tokens)
    np.testing.assert_array_equal(runs[0].logits, runs[1].logits)
    kv = make_kv(model, 32, 2, 64)
    one = run_stepwise(model, kv, prompts[1:2], 2, 12, 1.0, 8)
    # the same prompt in a smaller batch: the first-token logits are bit-identical
    # (later steps differ because the sample ids, and so the noise, differ)
    np.testing.assert_array_equal(one.logits[0], runs[0].logits[0][2:4])


@pytest.mark.parametrize("shape,n_prompts,G,P,steps", [(BF16_B, 3, 4, 100, 6), (BF16_A, 2, 8, 600, 4),
                                                       (BF16_A, 5, 3, 64, 3)])
def test_grouped_decode_bitexact_vs_per_row(shape, n_prompts, G, P, steps):
    """The prefix-shared decode kernel gives the same logits, bit for bit, as the per-row kernel,
    including a ragged group layout (groups of different sizes) and multi-split contexts."""
    w = synth.make_weights(shape, 5)
    wl = synth.Workload("t", shape, n_prompts, G, P, steps + 1)
    prompts = synth.make_prompts(wl, 5)
    model = engine.Model(shape, w)
    N = n_prompts * G
    kv = make_kv(model, 32, N, P + steps + 1)
    engine.prefill(model, kv, dev_i32(prompts), G, list(range(N)))
    shared = (P // 32) * 32
    rng = np.random.default_rng(0)
    for t in range(steps):
        L.dash_kv_reserve(kv.handle, list(range(N)), P + t + 1, engine.stream_handle())
        # drop a few rows (still grouped and in order) to exercise uneven groups
        keep = np.sort(rng.choice(N, size=N - (t % 3), replace=False)) if t else np.arange(N)
        toks = dev_i32(rng.integers(0, shape.vocab, keep.size))
        slots = dev_i32(keep)
        pos = dev_i32(np.full(keep.size, P + t))
        grp = keep // G
        off = np.concatenate([[0], np.flatnonzero(np.diff(grp)) + 1, [keep.size]]).astype(np.int32)
        # the per-row kernel first (it writes this step's K/V), then the grouped one
        # rewrites the same K/V values and must produce identical logits
        a = engine.decode_step(model, kv, toks, slots, pos).cpu().numpy()
        b = engine.decode_step_grouped(model, kv, toks, slots, pos, dev_i32(off), G, shared).cpu().numpy()
        np.testing.assert_array_equal(a, b)


@pytest.mark.parametrize("shape,n_prompts,G,P,steps", [(BF16_B, 2, 8, 600, 3), (BF16_A, 2, 4, 1100, 3)])
def test_grouped_decode_long_prefix_bitexact(shape, n_prompts, G, P, steps):
    """Prefix-shared decode over prompts longer than one LDS chunk of the prefix kernel
    (18 pages at head dim 128, 32 at head dim 64, 8 / 16 pages per chunk) in a cache whose
    slot count makes the split long enough to hold the whole prefix (and, at head dim 64,
    contexts that still need two splits): bit-identical to the per-row kernel."""
    w = synth.make_weights(shape, 6)
    wl = synth.Workload("t", shape, n_prompts, G, P, steps + 1)
    prompts = synth.make_prompts(wl, 6)
    model = engine.Model(shape, w)
    N = n_prompts * G
    ps, max_ctx = 32, P + steps + 8
    kv = engine.KVCache(model, ps, 1024, max_ctx, N * ((max_ctx + ps - 1) // ps) + 8)
    split = L.dash_kv_split_keys(kv.handle)
    assert split >= 512, split  # the whole shared prefix (or its first 512 keys) in split 0
    engine.prefill(model, kv, dev_i32(prompts), G, list(range(N)))
    shared = (P // ps) * ps
    off = dev_i32(np.arange(0, N + 1, G))
    rng = np.random.default_rng(1)
    for t in range(steps):
        L.dash_kv_reserve(kv.handle, list(range(N)), P + t + 1, engine.stream_handle())
        toks = dev_i32(rng.integers(0, shape.vocab, N))
        slots = dev_i32(np.arange(N))
        pos = dev_i32(np.full(N, P + t))
        a = engine.decode_step(model, kv, toks, slots, pos).cpu().numpy()
        b = engine.decode_step_grouped(model, kv, toks, slots, pos, off, G, shared).cpu().numpy()
        np.testing.assert_array_equal(a, b)


def test_grouped_decode_argument_errors():
    """dash_decode_step_grouped rejects, before any launch, groups above 8 rows, a shared
    length that is not a multiple of the page size or exceeds max_ctx, and bad group counts."""
    shape = BF16_B
    w = synth.make_weights(shape, 5)
    model = engine.Model(shape, w)
    kv = make_kv(model, 32, 8, 64)
    toks, slots, pos = dev_i32(np.zeros(8)), dev_i32(np.arange(8)), dev_i32(np.full(8, 40))
    off = dev_i32([0, 8])
    for group_size, shared, want in ((9, 32, L.DASH_ENOTSUP), (8, 20, L.DASH_EINVAL), (8, 96, L.DASH_EINVAL),
                                     (8, -32, L.DASH_EINVAL)):
        with pytest.raises(L.DashError) as e:
            engine.decode_step_grouped(model, kv, toks, slots, pos, off, group_size, shared)
        assert e.value.status == want, (group_size, shared)
    with pytest.raises(L.DashError) as e:  # more groups than rows
        engine.decode_step_grouped(model, kv, toks[:1], slots[:1], pos[:1], dev_i32([0, 1, 1]), 8, 32)
    assert e.value.status == L.DASH_EINVAL


def test_decode_halves_on_two_streams_bitexact():
    """Two halves of a batch decoded at the same time on two streams (separate workspaces,
    disjoint slots, shared prompt pages) give the full batch's logits bit for bit, at contexts
    that need several attention splits."""
    shape = BF16_A
    n_prompts, G, P, steps = 4, 4, 300, 3
    w = synth.make_weights(shape, 6)
    wl = synth.Workload("t", shape, n_prompts, G, P, steps + 1)
    prompts = synth.make_prompts(wl, 6)
    model = engine.Model(shape, w)
    N, H = n_prompts * G, n_prompts * G // 2
    kv = make_kv(model, 32, N, P + steps + 1)
    assert kv.split_keys < P  # the combine pass runs
    engine.prefill(model, kv, dev_i32(prompts), G, list(range(N)))
    wsa, wsb = model.workspace(H, kv.max_ctx), model.workspace(N - H, kv.max_ctx)
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    cur = torch.cuda.current_stream()
    rng = np.random.default_rng(1)
    for t in range(steps):
        L.dash_kv_reserve(kv.handle, list(range(N)), P + t + 1, engine.stream_handle())
        toks = dev_i32(rng.integers(0, shape.vocab, N))
        slots = dev_i32(np.arange(N))
        pos = dev_i32(np.full(N, P + t))
        full = engine.decode_step(model, kv, toks, slots, pos)
        la = torch.empty(H, shape.vocab, dtype=torch.float32, device="cuda")
        lb = torch.empty(N - H, shape.vocab, dtype=torch.float32, device="cuda")
        for st in (s1, s2):
            st.wait_stream(cur)
        # both halves rewrite this step's K/V with the values the full step wrote
        with torch.cuda.stream(s1):
            engine.decode_step(model, kv, toks[:H], slots[:H], pos[:H], wsa, la)
        with torch.cuda.stream(s2):
            engine.decode_step(model, kv, toks[H:], slots[H:], pos[H:], wsb, lb)
        cur.wait_stream(s1)
        cur.wait_stream(s2)
        np.testing.assert_array_equal(torch.cat([la, lb]).cpu().numpy(), full.cpu().numpy())


def test_rollout_driver_matches_stepwise_tiny():
    wl = synth.WORKLOADS["tiny"]
    w = synth.make_weights(wl.shape, 0)
    prompts = synth.make_prompts(wl, 0)
    model = engine.Model(wl.shape, w)
    kv = make_kv(model, 16, wl.n_seqs, wl.prompt_len + wl.gen_len)
    step = run_stepwise(model, kv, prompts, wl.group, wl.gen_len, 1.0, 2, keep_logits=False)
    ro = engine.Rollout(model, kv, wl.n_prompts, wl.prompt_len, wl.group, wl.gen_len)
    for use_graph in (False, True):
        toks, lps = ro.run(dev_i32(prompts), 1.0, 2, use_graph=use_graph)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(toks.cpu().numpy(), step.tokens)
        np.testing.assert_array_equal(lps.cpu().numpy(), step.logprobs)
    assert kv.free_pages == kv.pool.numel() // L.dash_kv_page_bytes(model.handle, 16)


def test_rollout_graph_profiling_times_every_launch():
    """Kernel-class timing under graph replay: each decode step's attention launches
    are event-record nodes of the graph; every replay is counted once, with the same
    tokens as an untimed run."""
    shape = BF16_A
    w = synth.make_weights(shape, 6)
    n_prompts, G, P, T = 2, 4, 70, 9
    prompts = synth.make_prompts(synth.Workload("t", shape, n_prompts, G, P, T), 6)
    model = engine.Model(shape, w)
    kv = make_kv(model, 32, n_prompts * G, P + T)
    ro = engine.Rollout(model, kv, n_prompts, P, G, T)
    plain, _ = ro.run(dev_i32(prompts), 1.0, 3, use_graph=True)
    plain = plain.cpu().numpy().copy()
    L.dash_profile_read(reset=True)
    L.dash_profile_enable((1 << L.K["attn"]) | (1 << L.K["sample"]))
    try:
        timed, _ = ro.run(dev_i32(prompts), 1.0, 3, use_graph=True)
        torch.cuda.synchronize()
        prof = L.dash_profile_read(reset=True)
    finally:
        L.dash_profile_enable(0)
    np.testing.assert_array_equal(timed.cpu().numpy(), plain)
    ms, n = prof["attn"]
    assert n == shape.n_layers * (T - 1) and ms > 0
    assert prof["sample"][1] == T - 1  # the first token is sampled outside the decode loop, untimed
    assert prof["gemm_qkv"][1] == 0
    # one layer's launches only
    L.dash_profile_enable(1 << L.K["attn"])
    L.dash_profile_layer(1)
    try:
        ro.run(dev_i32(prompts), 1.0, 3, use_graph=True)
        torch.cuda.synchronize()
        prof = L.dash_profile_read(reset=True)
    finally:
        L.dash_profile_enable(0)
        L.dash_profile_layer(-1)
    assert prof["attn"][1] == T - 1 and prof["attn"][0] > 0


@pytest.mark.parametrize("shape", [BF16_A, BF16_B])
def test_rollout_driver_ragged_and_graph_bf16(shape):
    w = synth.make_weights(shape, 4)
    n_prompts, G, P, T = 4, 4, 37, 40
    wl = synth.Workload("t", shape, n_prompts, G, P, T)
    prompts = synth.make_prompts(wl, 4)
    model = engine.Model(shape, w)
    kv = make_kv(model, 32, n_prompts * G, P + T)
    step = run_stepwise(model, kv, prompts, G, T, 1.0, 3)
    ro = engine.Rollout(model, kv, n_prompts, P, G, T)
    for use_graph in (False, True):
        toks, lps = ro.run(dev_i32(prompts), 1.0, 3, use_graph=use_graph)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(toks.cpu().numpy(), step.tokens)
    budgets = np.random.default_rng(0).integers(1, T + 1, n_prompts * G).astype(np.int32)
    budgets[0], budgets[1] = 1, T
    toks, lps = ro.run(dev_i32(prompts), 1.0, 3, budgets=budgets, use_graph=False)
    torch.cuda.synchronize()
    got = toks.cpu().numpy()
    for n in range(n_prompts * G):
        b = budgets[n]
        # batch-invariant kernels: a sample's tokens do not depend on which other rows are live
        np.testing.assert_array_equal(got[n, :b], step.tokens[n, :b])
        assert (got[n, b:] == -1).all()
    assert kv.free_pages == kv.pool.numel() // L.dash_kv_page_bytes(model.handle, 32)


def test_capacity_errors():
    shape = BF16_A
    model = engine.Model(shape, synth.make_weights(shape, 0))
    kv = engine.KVCache(model, 32, 4, 64, 3)
    pr = dev_i32(np.zeros((2, 40)))
    with pytest.raises(L.DashError) as e:  # 2 prompts x (1 full + 2 partial) pages > 3
        engine.prefill(model, kv, pr, 2, [0, 1, 2, 3])
    assert e.value.status == L.DASH_ECAPACITY
    assert kv.free_pages == 3
    with pytest.raises(L.DashError) as e:
        L.dash_kv_reserve(kv.handle, [0], 65, engine.stream_handle())
    assert e.value.status == L.DASH_ECAPACITY
    ws = model.workspace(2, 64)
    with pytest.raises(L.DashError) as e:
        L.dash_decode_step(model.handle, kv.handle, pr.data_ptr(), pr.data_ptr(), pr.data_ptr(), 4, pr.data_ptr(),
                           engine.aligned(ws), ws.numel() - 256, engine.stream_handle())
    assert e.value.status == L.DASH_ECAPACITY


def test_unbacked_position_sets_status_and_does_not_fault():
    shape = BF16_A
    model = engine.Model(shape, synth.make_weights(shape, 0))
    kv = make_kv(model, 32, 2, 64)
    L.dash_kv_reserve(kv.handle, [0], 10, engine.stream_handle())
    logits = engine.decode_step(model, kv, dev_i32([1, 2]), dev_i32([0, 1]), dev_i32([5, 5]))
    torch.cuda.synchronize()
    assert torch.isfinite(logits[0]).all()
    assert L.dash_kv_device_status(kv.handle, engine.stream_handle()) & 1
    assert L.dash_kv_device_status(kv.handle, engine.stream_handle()) == 0


def test_bad_token_sets_status_and_poisons_only_its_row():
    """A token outside [0, vocab) is never used as an index: its row's logits are NaN, the
    cache's status word gets DASH_ST_BAD_TOKEN, and the other rows' logits are bit-identical
    to a step in which every token was valid."""
    shape = BF16_A
    model = engine.Model(shape, synth.make_weights(shape, 0))
    kv = make_kv(model, 32, 3, 64)
    L.dash_kv_reserve(kv.handle, [0, 1, 2], 10, engine.stream_handle())
    slots, pos = dev_i32([0, 1, 2]), dev_i32([5, 5, 5])
    good = engine.decode_step(model, kv, dev_i32([1, 2, 3]), slots, pos).cpu().numpy()
    assert L.dash_kv_device_status(kv.handle, engine.stream_handle()) == 0
    bad = engine.decode_step(model, kv, dev_i32([1, -1, shape.vocab]), slots, pos).cpu().numpy()
    assert L.dash_kv_device_status(kv.handle, engine.stream_handle()) == L.DASH_ST_BAD_TOKEN
    np.testing.assert_array_equal(bad[0], good[0])
    assert np.isnan(bad[1:]).all()
    assert L.dash_kv_device_status(kv.handle, engine.stream_handle()) == 0


@pytest.mark.parametrize("shape,n_prompts,G,P,T", [(BF16_B, 2, 4, 100, 8), (BF16_A, 2, 8, 600, 4)])
def test_grouped_decode_matches_oracle(shape, n_prompts, G, P, T):
    """The prefix-shared decode kernel (each prompt's samples as one group over the prompt's
    full pages) against the oracle: logits within the bf16 tolerance at every generated
    position, and the oracle sampler reproduces the tokens from those logits."""
    w = synth.make_weights(shape, 15)
    wl = synth.Workload("t", shape, n_prompts, G, P, T)
    prompts = synth.make_prompts(wl, 15)
    model = engine.Model(shape, w)
    kv = make_kv(model, 32, n_prompts * G, P + T)
    run = run_stepwise(model, kv, prompts, G, T, 1.0, 19, grouped=True)
    worst = _check_run(shape, w, prompts, G, T, run, 1.0, 19, TOL[shape.dtype])
    print(f"grouped {shape.name} P={P}: max |dlogits| = {worst:.3g}")


@pytest.mark.parametrize("shape,P,T", [(BF16_B, 45, 24), (BF16_A, 33, 40)])
def test_stale_nonfinite_pool_bytes_do_not_change_results(shape, P, T):
    """Cache bytes past a row's context (the unused slots of its last page, pages never
    written) are never used: with every pool byte set to a bf16 NaN pattern before the
    prefill, the stepwise decode (per-row and prefix-shared attention), the graph-replayed
    rollout and the teacher-forced recompute give the same bits as with a zeroed pool.
    Contexts run through partial last pages (P, P + T not multiples of the page size),
    where the decode kernel skips the loads past the context and zeroes V there."""
    n_prompts, G = 2, 4
    N = n_prompts * G
    w = synth.make_weights(shape, 5)
    wl = synth.Workload("t", shape, n_prompts, G, P, T)
    prompts = synth.make_prompts(wl, 5)
    model = engine.Model(shape, w)

    def fresh_kv(nan: bool):
        kv = make_kv(model, 32, N, P + T)
        if nan:
            kv.pool.view(torch.int16).fill_(0x7FC0)
            torch.cuda.synchronize()
        return kv

    runs = {}
    for nan in (False, True):
        for grouped in (False, True):
            kv = fresh_kv(nan)
            runs[nan, grouped] = run_stepwise(model, kv, prompts, G, T, 1.0, 11, grouped=grouped)
            kv.close()
    for grouped in (False, True):
        a, b = runs[False, grouped], runs[True, grouped]
        np.testing.assert_array_equal(a.tokens, b.tokens)
        assert np.array_equal(a.logits.view(np.uint32), b.logits.view(np.uint32)), f"grouped={grouped}"
        assert np.array_equal(a.logprobs.view(np.uint32), b.logprobs.view(np.uint32))

    outs = {}
    for nan in (False, True):
        kv = fresh_kv(nan)
        ro = engine.Rollout(model, kv, n_prompts, P, G, T)
        toks, lps = ro.run(dev_i32(prompts), 1.0, 11, use_graph=True)
        seqs = torch.cat([dev_i32(np.repeat(prompts, G, axis=0)), toks], dim=1)
        kv.close()
        kv = fresh_kv(nan)
        tf = engine.teacher_forced_logprobs(model, kv, seqs, P)
        kv.close()
        outs[nan] = (toks.cpu().numpy(), lps.cpu().numpy(), tf.cpu().numpy())
    for x, y in zip(outs[False], outs[True]):
        assert np.array_equal(x.view(np.uint32), y.view(np.uint32))
    np.testing.assert_array_equal(outs[True][0], runs[True, False].tokens)
