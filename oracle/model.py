"""Oracle decoder forward pass (float64) — test infrastructure only.

The paper samples trajectories from the policy LM pi_theta (Sec. 3 problem
statement and Eq. (1)); it names Qwen2.5 base models (Sec. 4.1) and says
nothing else about the network.  This module writes out that network as the
plain definition, one sequence at a time, with a full causal recompute over the
whole (prompt + generated) sequence, so one call yields the next-token logits
at every position (teacher forcing).  Readings taken where the paper is silent:

* pre-norm decoder: x += Attn(RMSNorm(x)); x += MLP(RMSNorm(x)); logits =
  RMSNorm(x) E^T with the embedding E tied to the LM head;
* RMSNorm y = x / sqrt(mean(x^2) + eps) * w;
* q/k/v projections carry a bias, the output and MLP projections do not;
* rotate-half RoPE with frequencies theta^(-2i/hd), i < hd/2;
* grouped-query attention: query head h reads kv head h // (Hq/Hkv), scale
  1/sqrt(hd), causal softmax;
* SwiGLU MLP: down(silu(gate(y)) * up(y)), silu(z) = z / (1 + e^-z).

bfloat16 shapes (``dtype == 1``) round, exactly where the GPU path stores a
bfloat16 tensor, to the nearest bfloat16: every matmul left operand (the
normalised activations, the attention output, the SwiGLU product), q after
RoPE, and every cached key and value.  Everything else is float64.

Pins (tests/test_oracle_model.py): a library-routine reference built from
torch.nn.functional (rms_norm, scaled_dot_product_attention, silu, linear) with
RoPE written as complex multiplication; scalar-loop brute force on a micro
shape; the one-token closed form (attention over a single key returns its
value); RoPE identity at position 0, norm preservation and relative-position
invariance; causality (logits at position i do not depend on later tokens); and,
for the bfloat16 storage points, a scalar-loop brute force that rounds with
torch's own bfloat16 conversion at exactly those points (equal to the oracle,
while leaving out any single point moves the logits visibly).
"""
from __future__ import annotations

import numpy as np


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Nearest bfloat16 (ties to even) of float64 values, via float32; returns float64."""
    f = np.asarray(x, dtype=np.float64).astype(np.float32)
    b = f.view(np.uint32).astype(np.uint64)
    b = (b + 0x7FFF + ((b >> 16) & 1)) >> 16 << 16
    return b.astype(np.uint32).view(np.float32).astype(np.float64)


def as_f64(w: np.ndarray) -> np.ndarray:
    """Weight array (float32 values, or uint16 bfloat16 bit patterns) as float64."""
    w = np.asarray(w)
    if w.dtype == np.uint16:
        return (w.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return w.astype(np.float64)


def rmsnorm(x: np.ndarray, w: np.ndarray, eps: float) -> np.ndarray:
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * w


def rope_angles(pos: np.ndarray, hd: int, theta: float) -> tuple[np.ndarray, np.ndarray]:
    """cos and sin of pos * theta^(-2i/hd) for i < hd/2: arrays [len(pos), hd/2]."""
    i = np.arange(hd // 2, dtype=np.float64)
    freq = theta ** (-2.0 * i / hd)
    ang = np.asarray(pos, dtype=np.float64)[:, None] * freq[None, :]
    return np.cos(ang), np.sin(ang)


def rope(z: np.ndarray, cos: np.ndarray, sin: np.ndarray) -> np.ndarray:
    """Rotate-half RoPE of z [S, heads, hd] with per-position cos/sin [S, hd/2]."""
    h = z.shape[-1] // 2
    a, b = z[..., :h], z[..., h:]
    c, s = cos[:, None, :], sin[:, None, :]
    return np.concatenate([a * c - b * s, b * c + a * s], axis=-1)


def causal_gqa_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray) -> np.ndarray:
    """q [S, Hq, hd], k/v [S, Hkv, hd] -> o [S, Hq, hd]; causal, scale 1/sqrt(hd)."""
    S, Hq, hd = q.shape
    rep = Hq // k.shape[1]
    o = np.empty_like(q)
    mask = np.triu(np.ones((S, S), dtype=bool), 1)
    for h in range(Hq):
        kh, vh = k[:, h // rep, :], v[:, h // rep, :]
        s = (q[:, h, :] @ kh.T) / q.dtype.type(np.sqrt(hd))
        s[mask] = -np.inf
        s = s - s.max(axis=1, keepdims=True)
        p = np.exp(s)
        p /= p.sum(axis=1, keepdims=True)
        o[:, h, :] = p @ vh
    return o


def silu(z: np.ndarray) -> np.ndarray:
    return z / (1.0 + np.exp(-z))


def forward(shape: dict, weights: dict, tokens: np.ndarray,
            positions: np.ndarray | None = None, arith=np.float64) -> np.ndarray:
    """Next-token logits (float64) of one sequence.

    ``shape`` has keys n_layers, d_model, n_heads, n_kv_heads, head_dim, d_ff,
    vocab, rope_theta, rms_eps, dtype.  ``weights`` maps the tensor names
    embed, final_norm, l{i}.attn_norm, l{i}.w_qkv [(Hq+2Hkv)hd, d] (q rows, then
    k, then v), l{i}.b_qkv, l{i}.w_o [d, Hq hd], l{i}.mlp_norm,
    l{i}.w_gate_up [2 d_ff, d] (gate rows, then up rows), l{i}.w_down [d, d_ff].
    ``tokens`` int [S] occupy positions 0..S-1.  Returns logits [len(positions), V]
    at the requested positions (default: all).

    ``arith`` (float64 by default) is the floating-point type every operation is
    evaluated in.  float32 evaluates the same definition with float32 rounding; the
    tests use it only to measure how far fp32 arithmetic alone moves the logits of a
    deep bf16 network (through the bf16 storage points) from the float64 values.
    """
    bf = shape["dtype"] == 1
    A = arith
    rb = (lambda a: round_bf16(a).astype(A)) if bf else (lambda a: a)
    L, Hq, Hkv, hd = shape["n_layers"], shape["n_heads"], shape["n_kv_heads"], shape["head_dim"]
    ff, eps = shape["d_ff"], A(shape["rms_eps"])
    W = lambda name: as_f64(weights[name]).astype(A, copy=False)
    tokens = np.asarray(tokens)
    S = tokens.shape[0]
    E = W("embed")
    x = E[tokens].copy()
    cos, sin = rope_angles(np.arange(S), hd, shape["rope_theta"])
    cos, sin = cos.astype(A), sin.astype(A)
    for l in range(L):
        p = f"l{l}."
        y = rb(rmsnorm(x, W(p + "attn_norm"), eps))
        qkv = y @ W(p + "w_qkv").T + W(p + "b_qkv")
        q = qkv[:, :Hq * hd].reshape(S, Hq, hd)
        k = qkv[:, Hq * hd:(Hq + Hkv) * hd].reshape(S, Hkv, hd)
        v = qkv[:, (Hq + Hkv) * hd:].reshape(S, Hkv, hd)
        q = rb(rope(q, cos, sin))
        k = rb(rope(k, cos, sin))
        v = rb(v)
        o = rb(causal_gqa_attention(q, k, v).reshape(S, Hq * hd))
        x = x + o @ W(p + "w_o").T
        y = rb(rmsnorm(x, W(p + "mlp_norm"), eps))
        gu = y @ W(p + "w_gate_up").T
        h = rb(silu(gu[:, :ff]) * gu[:, ff:])
        x = x + h @ W(p + "w_down").T
    if positions is not None:
        x = x[np.asarray(positions)]
    y = rb(rmsnorm(x, W("final_norm"), eps))
    return (y @ E.T).astype(np.float64)


def rollout_logits(shape: dict, weights: dict, prompt: np.ndarray, generated: np.ndarray) -> np.ndarray:
    """Teacher-forced logits that produced each generated token.

    Token ``generated[t]`` was sampled from the logits at position P-1+t, where
    P = len(prompt).  Returns float64 [len(generated), V].
    """
    P, T = len(prompt), len(generated)
    seq = np.concatenate([np.asarray(prompt), np.asarray(generated)[:max(T - 1, 0)]])
    return forward(shape, weights, seq, positions=np.arange(P - 1, P - 1 + T))
