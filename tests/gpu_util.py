"""Helpers for the GPU parity tests: bring up the HIP path through the C ABI and
run prefill / decode / sample step by step, keeping every step's logits so the
oracle can check them."""
from __future__ import annotations

import dataclasses

import numpy as np
import pytest
import torch

from paper_2505_17218_amd import _lib as L
from paper_2505_17218_amd import engine, synth


def require_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    L.load()  # raises if libdash.so is missing: the GPU path has no fallback


def shape_dict(s: synth.Shape) -> dict:
    return dataclasses.asdict(s)


def dev_i32(a) -> torch.Tensor:
    return torch.as_tensor(np.asarray(a, dtype=np.int32)).cuda()


@dataclasses.dataclass
class StepRun:
    tokens: np.ndarray      # int32 [N, T]
    logprobs: np.ndarray    # float32 [N, T]
    logits: np.ndarray      # float32 [T, N, V] (logits each token was drawn from)


def run_stepwise(model: engine.Model, kv: engine.KVCache, prompts: np.ndarray, group: int, gen_len: int,
                 temperature: float, seed: int, keep_logits: bool = True, grouped: bool = False) -> StepRun:
    """Prefill, then gen_len - 1 decode steps, sampling after each; all through the C ABI.
    grouped: decode with dash_decode_step_grouped (each prompt's samples as one
    prefix-sharing group over the prompt's full pages)."""
    n_prompts, P = prompts.shape
    N = n_prompts * group
    V = model.shape.vocab
    pr = dev_i32(prompts)
    slots = list(range(N))
    logits0 = engine.prefill(model, kv, pr, group, slots)
    row_of = dev_i32(np.arange(N) // group)
    uid = dev_i32(np.arange(N))
    slot_t = dev_i32(np.arange(N))
    toks = np.zeros((N, gen_len), np.int32)
    lps = np.zeros((N, gen_len), np.float32)
    all_logits = np.zeros((gen_len, N, V), np.float32) if keep_logits else None
    tok, lp = engine.sample(logits0, uid, dev_i32(np.zeros(N)), temperature, seed, row_of=row_of)
    toks[:, 0] = tok.cpu().numpy()
    lps[:, 0] = lp.cpu().numpy()
    if keep_logits:
        all_logits[0] = logits0.cpu().numpy()[np.arange(N) // group]
    ws = model.workspace(N, kv.max_ctx)
    group_off = dev_i32(np.arange(0, N + 1, group))
    shared = P // kv.page_size * kv.page_size
    for t in range(1, gen_len):
        pos = P + t - 1
        engine.L.dash_kv_reserve(kv.handle, slots, pos + 1, engine.stream_handle())
        if grouped:
            logits = engine.decode_step_grouped(model, kv, tok, slot_t, dev_i32(np.full(N, pos)), group_off, group,
                                                shared, ws=ws)
        else:
            logits = engine.decode_step(model, kv, tok, slot_t, dev_i32(np.full(N, pos)), ws=ws)
        tok, lp = engine.sample(logits, uid, dev_i32(np.full(N, t)), temperature, seed)
        toks[:, t] = tok.cpu().numpy()
        lps[:, t] = lp.cpu().numpy()
        if keep_logits:
            all_logits[t] = logits.cpu().numpy()
    torch.cuda.synchronize()
    L.dash_kv_release(kv.handle, slots)
    return StepRun(toks, lps, all_logits)


def make_kv(model: engine.Model, page_size: int, max_seqs: int, max_ctx: int, extra_pages: int = 8):
    pages_per_seq = (max_ctx + page_size - 1) // page_size
    return engine.KVCache(model, page_size, max_seqs, max_ctx, max_seqs * pages_per_seq + extra_pages)


def kl_sensitivity(la: np.ndarray, lb: np.ndarray):
    """First-order bounds of |d KL| per unit max-norm change of the logits, per row, for
    D_KL(b || a): sum |p_a - p_b| (through a) + E_b |log(p_b / p_a) - KL| (through b);
    and the reverse direction with the roles swapped.  A GPU KL computed from logits within
    delta of the float64 ones lies within about delta times this of the exact KL."""
    la = np.asarray(la, dtype=np.float64)
    lb = np.asarray(lb, dtype=np.float64)
    lsa = la - (la.max(1, keepdims=True) + np.log(np.exp(la - la.max(1, keepdims=True)).sum(1, keepdims=True)))
    lsb = lb - (lb.max(1, keepdims=True) + np.log(np.exp(lb - lb.max(1, keepdims=True)).sum(1, keepdims=True)))
    pa, pb = np.exp(lsa), np.exp(lsb)
    kl = np.sum(pb * (lsb - lsa), 1)
    kl_rev = np.sum(pa * (lsa - lsb), 1)
    tv2 = np.abs(pa - pb).sum(1)
    return tv2 + np.sum(pb * np.abs(lsb - lsa - kl[:, None]), 1), tv2 + np.sum(pa * np.abs(lsa - lsb - kl_rev[:, None]), 1)
