"""Seeded synthetic inputs for DASH rollouts: decoder shapes, random-init weights,
prompts, rewards and ragged generation lengths.

This module draws random numbers and lays them out; it computes nothing of the
method itself (no forward pass, no sampling, no advantage).  It is the one
module that both the HIP path and the oracle consume, so that both see exactly
the same inputs.

Seeding (run seed ``s``): weights use sub-seed ``s+0``, prompts ``s+1``, the
sampler key ``s+2``, rewards ``s+3`` and ragged lengths ``s+4``.

Stand-in data: the paper trains on MATH/MBPP+ prompts with binary verifier
rewards (Sec. 4.1, Sec. 3 problem statement) and Qwen2.5 base weights.  None of
that is used here; uniform token ids, N(0, 0.02) weights and Bernoulli rewards
with the same shapes stand in for them.
"""
from __future__ import annotations

import dataclasses
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

DT_F32 = 0
DT_BF16 = 1


@dataclasses.dataclass(frozen=True)
class Shape:
    """Decoder shape (a Qwen2.5-style pre-norm GQA decoder with tied embeddings)."""
    name: str
    n_layers: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    d_ff: int
    vocab: int
    rope_theta: float
    dtype: int  # DT_F32 or DT_BF16
    rms_eps: float = 1e-6

    @property
    def qkv_rows(self) -> int:
        return (self.n_heads + 2 * self.n_kv_heads) * self.head_dim

    @property
    def n_params(self) -> int:
        d, hd = self.d_model, self.head_dim
        per_layer = (2 * d + self.qkv_rows * d + self.qkv_rows
                     + d * self.n_heads * hd + 3 * self.d_ff * d)
        return self.vocab * d + d + self.n_layers * per_layer


@dataclasses.dataclass(frozen=True)
class Workload:
    """A rollout workload: shape, prompt groups, generation budget, rewards."""
    name: str
    shape: Shape
    n_prompts: int
    group: int
    prompt_len: int
    gen_len: int                  # tokens generated per sample (cap for ragged)
    temperature: float = 1.0
    reward: str = "bernoulli0.5"  # or "beta0.5"
    ragged_mean: float = 0.0      # >0: geometric lengths with this mean, capped at gen_len
    tau: float = 0.1

    @property
    def n_seqs(self) -> int:
        return self.n_prompts * self.group


TINY = Shape("tiny", 2, 64, 4, 2, 16, 172, 512, 10000.0, DT_F32)
QWEN05 = Shape("qwen2.5-0.5b", 24, 896, 14, 2, 64, 4864, 151936, 1e6, DT_BF16)
QWEN15 = Shape("qwen2.5-1.5b", 28, 1536, 12, 2, 128, 8960, 151936, 1e6, DT_BF16)
QWEN3 = Shape("qwen2.5-3b", 36, 2048, 16, 2, 128, 11008, 151936, 1e6, DT_BF16)

WORKLOADS = {
    "tiny": Workload("tiny", TINY, 4, 4, 16, 32),
    "0.5b-b512": Workload("0.5b-b512", QWEN05, 64, 8, 256, 1024, reward="beta0.5"),
    "1.5b-b1024": Workload("1.5b-b1024", QWEN15, 128, 8, 256, 1024, reward="beta0.5"),
    "3b-b64": Workload("3b-b64", QWEN3, 8, 8, 512, 1024, reward="beta0.5"),
    "3b-b256": Workload("3b-b256", QWEN3, 32, 8, 512, 1024, reward="beta0.5"),
    "3b-b1024": Workload("3b-b1024", QWEN3, 128, 8, 512, 1024, reward="beta0.5"),
    "3b-b2048": Workload("3b-b2048", QWEN3, 256, 8, 512, 1024, reward="beta0.5"),
    "1.5b-ragged": Workload("1.5b-ragged", QWEN15, 512, 8, 256, 2048, reward="beta0.5",
                            ragged_mean=600.0),
}


def weight_names(shape: Shape) -> list[str]:
    """Flat tensor order of the weight table (same order as the C ABI's table)."""
    names = ["embed", "final_norm", "lm_head"]
    for l in range(shape.n_layers):
        names += [f"l{l}.attn_norm", f"l{l}.w_qkv", f"l{l}.b_qkv", f"l{l}.w_o",
                  f"l{l}.mlp_norm", f"l{l}.w_gate_up", f"l{l}.w_down"]
    return names


def weight_shapes(shape: Shape) -> dict[str, tuple[int, ...]]:
    d, hd = shape.d_model, shape.head_dim
    out = {"embed": (shape.vocab, d), "final_norm": (d,), "lm_head": (0,)}
    for l in range(shape.n_layers):
        out[f"l{l}.attn_norm"] = (d,)
        out[f"l{l}.w_qkv"] = (shape.qkv_rows, d)
        out[f"l{l}.b_qkv"] = (shape.qkv_rows,)
        out[f"l{l}.w_o"] = (d, shape.n_heads * hd)
        out[f"l{l}.mlp_norm"] = (d,)
        out[f"l{l}.w_gate_up"] = (2 * shape.d_ff, d)
        out[f"l{l}.w_down"] = (d, shape.d_ff)
    return out


_CHUNK = 1 << 22


def _to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even); return the 16-bit patterns."""
    b = x.view(np.uint32)
    r = (b + np.uint32(0x7FFF) + ((b >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return r.astype(np.uint16)


def _fill_normal(out: np.ndarray, seed: int, tidx: int, bf16: bool, c: int) -> None:
    lo = c * _CHUNK
    hi = min(out.size, lo + _CHUNK)
    rng = np.random.default_rng([seed, tidx, c])
    v = rng.standard_normal(hi - lo, dtype=np.float32) * np.float32(0.02)
    if bf16:
        out[lo:hi] = _to_bf16_bits(v)
    else:
        out[lo:hi] = v


def make_weights(shape: Shape, seed: int = 0, threads: int | None = None) -> dict[str, np.ndarray]:
    """Random-init weights: every matrix, the embedding and the q/k/v bias are
    N(0, 0.02); norm weights are 1.  Embeddings are tied (``lm_head`` is empty).

    bf16 shapes return uint16 arrays holding bfloat16 bit patterns (values
    rounded to nearest-even from the float32 draw); fp32 shapes return float32.
    Tensor ``i`` of :func:`weight_names`, flat chunk ``c`` (2^22 elements) is
    drawn from ``default_rng([seed, i, c])``, so the result is independent of
    the thread count.
    """
    bf16 = shape.dtype == DT_BF16
    dt = np.uint16 if bf16 else np.float32
    one = np.uint16(0x3F80) if bf16 else np.float32(1.0)
    shapes = weight_shapes(shape)
    out: dict[str, np.ndarray] = {}
    jobs = []
    for i, name in enumerate(weight_names(shape)):
        shp = shapes[name]
        arr = np.empty(int(np.prod(shp)), dtype=dt)
        if name.endswith("norm"):
            arr[:] = one
        elif arr.size:
            for c in range((arr.size + _CHUNK - 1) // _CHUNK):
                jobs.append((arr, i, c))
        out[name] = arr.reshape(shp)
    nthr = threads or min(16, len(os.sched_getaffinity(0)))
    with ThreadPoolExecutor(max_workers=nthr) as ex:
        list(ex.map(lambda j: _fill_normal(j[0], seed, j[1], bf16, j[2]), jobs))
    return out


def make_prompts(wl: Workload, seed: int = 0) -> np.ndarray:
    """Prompt token ids, uniform in [0, vocab): int32 [n_prompts, prompt_len]."""
    rng = np.random.default_rng(seed + 1)
    return rng.integers(0, wl.shape.vocab, size=(wl.n_prompts, wl.prompt_len), dtype=np.int32)


def sampler_seed(seed: int = 0) -> int:
    return seed + 2


def make_rewards(n_groups: int, group: int, kind: str = "bernoulli0.5", seed: int = 0) -> np.ndarray:
    """Binary rewards, float32 [n_groups * group] (groups contiguous).

    ``bernoulli0.5``: each sample independently Bernoulli(0.5).
    ``beta0.5``: per group p ~ Beta(0.5, 0.5), then each sample Bernoulli(p).
    """
    rng = np.random.default_rng(seed + 3)
    if kind == "bernoulli0.5":
        r = rng.random(n_groups * group) < 0.5
    elif kind == "beta0.5":
        p = rng.beta(0.5, 0.5, size=n_groups)
        r = (rng.random((n_groups, group)) < p[:, None]).reshape(-1)
    else:
        raise ValueError(kind)
    return r.astype(np.float32)


def make_lengths(n: int, mean: float, cap: int, seed: int = 0) -> np.ndarray:
    """Ragged generation lengths: Geometric(1/mean) on {1, 2, ...}, capped at ``cap``; int32 [n]."""
    rng = np.random.default_rng(seed + 4)
    return np.minimum(rng.geometric(1.0 / mean, size=n), cap).astype(np.int32)


def make_logits(rows: int, vocab: int, seed: int = 0, scale: float = 1.0) -> np.ndarray:
    """Random float32 logits [rows, vocab] ~ N(0, scale^2), for sampler tests."""
    rng = np.random.default_rng([seed, 7])
    return (rng.standard_normal((rows, vocab), dtype=np.float32) * np.float32(scale))
