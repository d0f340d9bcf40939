"""The allocation-free decode step (dash_decode_step_noalloc: the workspace is a device
array inside the library) against dash_decode_step with a caller workspace: the same
logits bit for bit on two calls in a row, the second with fewer rows, and a clear
capacity error for a batch whose workspace exceeds the array."""
import numpy as np
import pytest
import torch

from paper_2505_17218_amd import _lib as L
from paper_2505_17218_amd import engine, synth

from gpu_util import dev_i32, make_kv, require_gpu

pytestmark = pytest.mark.gpu

SHAPE = synth.Shape("bf16-noalloc", 2, 384, 6, 2, 128, 768, 2051, 1e6, synth.DT_BF16)
SCRATCH_BYTES = 64 << 20


def test_noalloc_decode_matches_decode_step():
    require_gpu()
    w = synth.make_weights(SHAPE, 31)
    n_prompts, G, P = 6, 4, 70
    prompts = synth.make_prompts(synth.Workload("t", SHAPE, n_prompts, G, P, 4), 31)
    model = engine.Model(SHAPE, w)
    N = n_prompts * G
    kv = make_kv(model, 32, N, P + 4)
    engine.prefill(model, kv, dev_i32(prompts), G, list(range(N)))
    st = engine.stream_handle()
    rng = np.random.default_rng(2)
    for t, rows in ((0, N), (1, N // 2 - 1)):  # two calls in a row, the second with fewer rows
        L.dash_kv_reserve(kv.handle, list(range(rows)), P + t + 1, st)
        toks = dev_i32(rng.integers(0, SHAPE.vocab, rows))
        slots, pos = dev_i32(np.arange(rows)), dev_i32(np.full(rows, P + t))
        want = engine.decode_step(model, kv, toks, slots, pos).cpu().numpy()
        got = torch.full((rows, SHAPE.vocab), float("nan"), dtype=torch.float32, device="cuda")
        L.dash_decode_step_noalloc(model.handle, kv.handle, toks.data_ptr(), slots.data_ptr(), pos.data_ptr(), rows,
                                   got.data_ptr(), st)
        np.testing.assert_array_equal(got.cpu().numpy(), want)
    assert L.dash_kv_device_status(kv.handle, st) == 0
    # a batch whose workspace exceeds the array is refused before any launch
    big = 1
    while L.dash_workspace_bytes(model.handle, big, kv.max_ctx) <= SCRATCH_BYTES:
        big *= 2
    with pytest.raises(L.DashError) as e:
        L.dash_decode_step_noalloc(model.handle, kv.handle, toks.data_ptr(), slots.data_ptr(), pos.data_ptr(), big,
                                   got.data_ptr(), st)
    assert e.value.status == L.DASH_ECAPACITY
