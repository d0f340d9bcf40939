"""Pins for the oracle decoder forward pass (oracle/model.py)."""
import dataclasses
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import model as om
from paper_2505_17218_amd import synth


def _shape(s: synth.Shape) -> dict:
    return dataclasses.asdict(s)


MICRO = synth.Shape("micro", 2, 8, 4, 2, 4, 12, 16, 10000.0, synth.DT_F32)


def _torch_reference(shape: dict, weights: dict, tokens: np.ndarray) -> np.ndarray:
    """Independent formulation from library routines: F.rms_norm, F.linear,
    F.scaled_dot_product_attention (causal), F.silu, and RoPE as a complex
    rotation (z_i + j z_{i+hd/2}) * exp(j p w_i)."""
    t = lambda a: torch.from_numpy(om.as_f64(a))
    L, Hq, Hkv, hd = shape["n_layers"], shape["n_heads"], shape["n_kv_heads"], shape["head_dim"]
    ff, eps, d = shape["d_ff"], shape["rms_eps"], shape["d_model"]
    tok = torch.from_numpy(np.asarray(tokens, dtype=np.int64))
    S = tok.numel()
    E = t(weights["embed"])
    x = E[tok]
    pos = torch.arange(S, dtype=torch.float64)
    w = shape["rope_theta"] ** (-torch.arange(0, hd, 2, dtype=torch.float64) / hd)
    rot = torch.polar(torch.ones(S, hd // 2, dtype=torch.float64), pos[:, None] * w[None, :])

    def rope(z):  # z [S, H, hd]
        zc = torch.complex(z[..., : hd // 2], z[..., hd // 2:]) * rot[:, None, :]
        return torch.cat([zc.real, zc.imag], dim=-1)

    for l in range(L):
        p = f"l{l}."
        y = F.rms_norm(x, (d,), t(weights[p + "attn_norm"]), eps)
        qkv = F.linear(y, t(weights[p + "w_qkv"]), t(weights[p + "b_qkv"]))
        q, k, v = torch.split(qkv, [Hq * hd, Hkv * hd, Hkv * hd], dim=-1)
        q = rope(q.reshape(S, Hq, hd))
        k = rope(k.reshape(S, Hkv, hd))
        v = v.reshape(S, Hkv, hd)
        k = k.repeat_interleave(Hq // Hkv, dim=1)
        v = v.repeat_interleave(Hq // Hkv, dim=1)
        o = F.scaled_dot_product_attention(q.transpose(0, 1), k.transpose(0, 1), v.transpose(0, 1),
                                           is_causal=True)
        x = x + F.linear(o.transpose(0, 1).reshape(S, Hq * hd), t(weights[p + "w_o"]))
        y = F.rms_norm(x, (d,), t(weights[p + "mlp_norm"]), eps)
        g, u = torch.split(F.linear(y, t(weights[p + "w_gate_up"])), [ff, ff], dim=-1)
        x = x + F.linear(F.silu(g) * u, t(weights[p + "w_down"]))
    y = F.rms_norm(x, (d,), t(weights["final_norm"]), eps)
    return F.linear(y, E).numpy()


def _brute(shape: dict, weights: dict, tokens, rnd=None) -> np.ndarray:
    """Scalar loops over every index (micro shapes only).  ``rnd(point, values)``, if given,
    is applied to the list of values at each named storage point (see BF16_POINTS)."""
    W = {k: om.as_f64(v) for k, v in weights.items()}
    R = rnd or (lambda point, vals: vals)
    L, Hq, Hkv, hd = shape["n_layers"], shape["n_heads"], shape["n_kv_heads"], shape["head_dim"]
    ff, eps, d, V = shape["d_ff"], shape["rms_eps"], shape["d_model"], shape["vocab"]
    S = len(tokens)
    x = [[W["embed"][tokens[s]][i] for i in range(d)] for s in range(S)]

    def norm(row, w):
        ms = sum(a * a for a in row) / d
        r = 1.0 / math.sqrt(ms + eps)
        return [row[i] * r * w[i] for i in range(d)]

    def lin(row, M, b=None):
        return [sum(M[n][kk] * row[kk] for kk in range(len(row))) + (b[n] if b is not None else 0.0)
                for n in range(len(M))]

    def rot(vec, s):
        h = hd // 2
        out = list(vec)
        for i in range(h):
            a = s * shape["rope_theta"] ** (-2.0 * i / hd)
            c, sn = math.cos(a), math.sin(a)
            out[i] = vec[i] * c - vec[i + h] * sn
            out[i + h] = vec[i + h] * c + vec[i] * sn
        return out

    for l in range(L):
        p = f"l{l}."
        qs, ks, vs = [], [], []
        for s in range(S):
            qkv = lin(R("attn_in", norm(x[s], W[p + "attn_norm"])), W[p + "w_qkv"], W[p + "b_qkv"])
            qs.append([R("q", rot(qkv[h * hd:(h + 1) * hd], s)) for h in range(Hq)])
            ks.append([R("k", rot(qkv[(Hq + h) * hd:(Hq + h + 1) * hd], s)) for h in range(Hkv)])
            vs.append([R("v", qkv[(Hq + Hkv + h) * hd:(Hq + Hkv + h + 1) * hd]) for h in range(Hkv)])
        for s in range(S):
            o = []
            for h in range(Hq):
                g = h // (Hq // Hkv)
                sc = [sum(qs[s][h][i] * ks[j][g][i] for i in range(hd)) / math.sqrt(hd) for j in range(s + 1)]
                m = max(sc)
                e = [math.exp(a - m) for a in sc]
                z = sum(e)
                o += [sum(e[j] / z * vs[j][g][i] for j in range(s + 1)) for i in range(hd)]
            x[s] = [a + b for a, b in zip(x[s], lin(R("attn_out", o), W[p + "w_o"]))]
        for s in range(S):
            gu = lin(R("mlp_in", norm(x[s], W[p + "mlp_norm"])), W[p + "w_gate_up"])
            hh = [gu[i] / (1.0 + math.exp(-gu[i])) * gu[ff + i] for i in range(ff)]
            x[s] = [a + b for a, b in zip(x[s], lin(R("swiglu", hh), W[p + "w_down"]))]
    return np.array([lin(R("final_in", norm(x[s], W["final_norm"])), W["embed"]) for s in range(S)])


@pytest.fixture(scope="module")
def micro():
    w = synth.make_weights(MICRO, seed=3)
    # non-trivial norm weights so that a dropped norm scale is visible
    rng = np.random.default_rng(11)
    for k in w:
        if k.endswith("norm"):
            w[k] = (1.0 + 0.5 * rng.standard_normal(w[k].shape)).astype(np.float32)
        elif w[k].size:
            w[k] = (w[k] * 25).astype(np.float32)  # O(0.5) weights: large logits differences
    return _shape(MICRO), w


def test_micro_matches_scalar_brute_force(micro):
    shape, w = micro
    toks = np.array([3, 1, 4, 1, 5, 9, 2], dtype=np.int32)
    got = om.forward(shape, w, toks)
    ref = _brute(shape, w, list(toks))
    np.testing.assert_allclose(got, ref, rtol=1e-10, atol=1e-10)


def test_micro_matches_torch_library_reference(micro):
    shape, w = micro
    toks = np.array([0, 15, 7, 7, 2, 11, 3, 8, 1, 12], dtype=np.int32)
    np.testing.assert_allclose(om.forward(shape, w, toks), _torch_reference(shape, w, toks),
                               rtol=1e-10, atol=1e-10)


def test_tiny_matches_torch_library_reference():
    shape = _shape(synth.TINY)
    w = synth.make_weights(synth.TINY, seed=0)
    toks = np.random.default_rng(5).integers(0, 512, size=40).astype(np.int32)
    np.testing.assert_allclose(om.forward(shape, w, toks), _torch_reference(shape, w, toks),
                               rtol=1e-9, atol=1e-12)


def test_bf16_shape_matches_reference_up_to_rounding_points():
    """A bf16 shape without the rounding points is the plain float64 network; with them
    it differs by about bf16 precision, not more."""
    s = synth.Shape("bf16-small", 2, 128, 4, 2, 32, 256, 300, 1e6, synth.DT_BF16)
    shape = _shape(s)
    w = synth.make_weights(s, seed=1)
    toks = np.random.default_rng(2).integers(0, 300, size=24).astype(np.int32)
    ref = _torch_reference(shape, w, toks)
    exact = om.forward(dict(shape, dtype=0), w, toks)
    np.testing.assert_allclose(exact, ref, rtol=1e-9, atol=1e-12)
    got = om.forward(shape, w, toks)
    err = np.abs(got - ref).max()
    assert 1e-5 < err < 2e-2, err


# Storage points where the bfloat16 path keeps bfloat16 values: the normalised input of the
# QKV projection, q and k after RoPE, v (the cached keys and values), the attention output
# (left operand of the output projection), the normalised MLP input, the SwiGLU product
# (left operand of the down projection) and the normalised input of the LM head.
BF16_POINTS = ("attn_in", "q", "k", "v", "attn_out", "mlp_in", "swiglu", "final_in")
MICRO_BF16 = synth.Shape("micro-bf16", 2, 8, 4, 2, 4, 12, 16, 10000.0, synth.DT_BF16)


def _torch_bf16(vals):
    """Nearest bfloat16 by torch's own conversion (a library routine, not the oracle's bit trick)."""
    return torch.tensor(vals, dtype=torch.float64).to(torch.bfloat16).to(torch.float64).tolist()


@pytest.fixture(scope="module")
def micro_bf16():
    w = synth.make_weights(MICRO_BF16, seed=4)
    rng = np.random.default_rng(12)
    for k in w:
        if k.endswith("norm"):
            v = (1.0 + 0.5 * rng.standard_normal(w[k].shape)).astype(np.float32)
        elif w[k].size:
            v = (om.as_f64(w[k]) * 25).astype(np.float32)  # O(0.5) weights
        else:
            continue
        w[k] = synth._to_bf16_bits(v)
    return _shape(MICRO_BF16), w


def test_bf16_rounding_points_pinned_by_brute_force(micro_bf16):
    """The bfloat16 oracle equals a scalar-loop brute force that rounds (with torch's
    conversion) at exactly the eight storage points; leaving out any one of them moves the
    logits by far more than the agreement, so a missing, extra or misplaced rounding point
    in the oracle fails here."""
    shape, w = micro_bf16
    toks = [3, 1, 4, 1, 5, 9, 2, 6, 5, 3]
    got = om.forward(shape, w, np.array(toks, dtype=np.int32))
    full = _brute(shape, w, toks, rnd=lambda point, vals: _torch_bf16(vals))
    np.testing.assert_allclose(got, full, rtol=1e-9, atol=1e-9)
    for skip in BF16_POINTS:
        part = _brute(shape, w, toks, rnd=lambda point, vals, skip=skip: vals if point == skip else _torch_bf16(vals))
        assert np.abs(part - got).max() > 1e-3, skip
    # and the float32 network (no rounding at all) is the dtype-0 oracle on the same weights
    np.testing.assert_allclose(om.forward(dict(shape, dtype=0), w, np.array(toks, dtype=np.int32)),
                               _brute(shape, w, toks), rtol=1e-10, atol=1e-10)


def test_causal_prefix_consistency(micro):
    """Logits at position i depend only on tokens 0..i (a KV-cached decode sees the same)."""
    shape, w = micro
    toks = np.array([5, 6, 7, 8, 9, 10, 11, 12], dtype=np.int32)
    full = om.forward(shape, w, toks)
    for i in range(1, len(toks) + 1):
        np.testing.assert_allclose(om.forward(shape, w, toks[:i])[-1], full[i - 1], rtol=1e-12, atol=1e-12)


def test_single_token_attention_returns_value(micro):
    """With one key, attention returns that key's value for every query head."""
    rng = np.random.default_rng(0)
    q = rng.standard_normal((1, 4, 8))
    k = rng.standard_normal((1, 2, 8))
    v = rng.standard_normal((1, 2, 8))
    o = om.causal_gqa_attention(q, k, v)
    np.testing.assert_allclose(o[0], v[0][[0, 0, 1, 1]], rtol=0, atol=0)


def test_gqa_head_mapping_and_mha_special_case():
    rng = np.random.default_rng(1)
    S, hd = 6, 8
    q = rng.standard_normal((S, 4, hd))
    k = rng.standard_normal((S, 2, hd))
    v = rng.standard_normal((S, 2, hd))
    o = om.causal_gqa_attention(q, k, v)
    o_mha = om.causal_gqa_attention(q, np.repeat(k, 2, axis=1), np.repeat(v, 2, axis=1))
    np.testing.assert_allclose(o, o_mha, rtol=1e-14, atol=1e-14)
    # head 1 must read kv head 0, head 2 kv head 1
    o_swap = om.causal_gqa_attention(q, k[:, ::-1], v[:, ::-1])
    assert not np.allclose(o[:, 1], o_swap[:, 1])


def test_rope_invariants():
    rng = np.random.default_rng(2)
    hd = 16
    z = rng.standard_normal((5, 3, hd))
    c, s = om.rope_angles(np.zeros(5), hd, 1e4)
    np.testing.assert_array_equal(om.rope(z, c, s), z)            # position 0 is the identity
    c, s = om.rope_angles(np.arange(5) * 37, hd, 1e4)
    r = om.rope(z, c, s)
    np.testing.assert_allclose(np.linalg.norm(r, axis=-1), np.linalg.norm(z, axis=-1), rtol=1e-13)
    # <R_m q, R_n k> depends on m - n only
    qv, kv = rng.standard_normal(hd), rng.standard_normal(hd)

    def dot(m, n):
        cm, sm = om.rope_angles(np.array([m]), hd, 1e4)
        cn, sn = om.rope_angles(np.array([n]), hd, 1e4)
        return float((om.rope(qv[None, None], cm, sm) * om.rope(kv[None, None], cn, sn)).sum())

    assert abs(dot(10, 3) - dot(107, 100)) < 1e-10
    assert abs(dot(10, 3) - dot(3, 10)) > 1e-6


def test_rmsnorm_and_silu_library():
    rng = np.random.default_rng(3)
    x = rng.standard_normal((4, 10))
    w = rng.standard_normal(10)
    ref = F.rms_norm(torch.from_numpy(x), (10,), torch.from_numpy(w), 1e-6).numpy()
    np.testing.assert_allclose(om.rmsnorm(x, w, 1e-6), ref, rtol=1e-13)
    np.testing.assert_allclose(om.silu(x), F.silu(torch.from_numpy(x)).numpy(), rtol=1e-13)
    # constant vector normalises to the norm weight
    np.testing.assert_allclose(om.rmsnorm(np.full((1, 10), 3.0), w, 0.0)[0], w, rtol=1e-15)


def test_zero_mlp_weights_leave_residual(micro):
    shape, w = micro
    w2 = dict(w)
    for l in range(shape["n_layers"]):
        w2[f"l{l}.w_down"] = np.zeros_like(w[f"l{l}.w_down"])
        w2[f"l{l}.w_o"] = np.zeros_like(w[f"l{l}.w_o"])
    toks = np.array([1, 2, 3], dtype=np.int32)
    E = om.as_f64(w["embed"])
    y = om.rmsnorm(E[toks], om.as_f64(w["final_norm"]), shape["rms_eps"])
    np.testing.assert_allclose(om.forward(shape, w2, toks), y @ E.T, rtol=1e-13)


def test_round_bf16_ties_to_even_and_exact_values():
    vals = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, 1.0 + 2 ** -9, -2.5, 0.0])
    want = np.array([1.0, 1.0, 1.0 + 4 * 2 ** -8, 1.0, -2.5, 0.0])
    np.testing.assert_array_equal(om.round_bf16(vals), want)


def test_rollout_logits_positions(micro):
    shape, w = micro
    prompt = np.array([1, 2, 3, 4], dtype=np.int32)
    gen = np.array([5, 6, 7], dtype=np.int32)
    lg = om.rollout_logits(shape, w, prompt, gen)
    full = om.forward(shape, w, np.concatenate([prompt, gen]))
    np.testing.assert_allclose(lg, full[3:6], rtol=1e-13)


def test_float32_arithmetic_mode(micro):
    """The float32 evaluation mode computes the same definition: on the float32 micro shape
    it agrees with the float64 evaluation to float32 precision, keeps float32 intermediates
    (so it is not float64 in disguise), and leaves the float64 default untouched."""
    shape, w = micro
    toks = np.array([3, 1, 4, 1, 5, 9, 2], dtype=np.int32)
    a64 = om.forward(shape, w, toks)
    a32 = om.forward(shape, w, toks, arith=np.float32)
    assert a32.dtype == np.float64
    np.testing.assert_allclose(a32, a64, rtol=2e-5, atol=2e-5)
    assert np.abs(a32 - a64).max() > 1e-9
    np.testing.assert_array_equal(om.forward(shape, w, toks, arith=np.float64), a64)
