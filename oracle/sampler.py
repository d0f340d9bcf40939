"""Oracle temperature sampler (float32, bit-exact contract) — test infrastructure only.

DASH draws G trajectories per prompt from the current policy (Sec. 3.4,
preemptive sampling; Sec. 3 problem statement: y ~ pi_theta(. | x)).  With
pure temperature sampling at temperature T, each token is a draw from
softmax(l / T).  This module draws it by the Gumbel-max method: with
independent standard Gumbel noise g_v, argmax_v (l_v / T + g_v) is distributed
as softmax(l / T).

The noise is counter-based so that a draw depends only on (seed, sample id,
step, vocab index), never on batch position or thread schedule:

1. key = (seed mod 2^32, seed >> 32); counter = (v >> 2, step, seq_uid, 0).
2. x = Philox4x32-10(counter, key) word (v & 3) — Salmon, Moraes, Dror and
   Shaw, "Parallel random numbers: as easy as 1, 2, 3" (SC'11): ten rounds of
   two 32x32->64 multiplies with the round-key bumped by the Weyl constants.
3. u = ((x >> 8) | 1) * 2^-24, exactly representable, in (0, 1).
4. g = -L(-L(u)), where L is the natural log defined by :func:`own_log`.
5. s_v = l_v / T + g_v (for T == 1 the division is skipped), float32.
6. token = argmax s_v over finite l_v, ties to the smallest v; -1 if no l_v is finite.

Every step is float32 IEEE arithmetic with each operation rounded on its own
(no fused multiply-add), so the GPU reproduces the token ids bit for bit from
the same logits.  The log-probability of the drawn token under softmax(l / T)
is computed here in float64 (it is compared with a tolerance, not bitwise).

Pins (tests/test_oracle_sampler.py): Philox against rocRAND's
philox4x32_10 engine compiled for the host; own_log against numpy's float64
log (<= 2 ulp); Gumbel mean/variance against the Euler-Mascheroni constant and
pi^2/6; chi-square of token frequencies against softmax(l/T); the uniform case
for constant logits; and the T -> 0 limit reducing to argmax.
"""
from __future__ import annotations

import math

import numpy as np

_M0, _M1 = np.uint64(0xD2511F53), np.uint64(0xCD9E8D57)
_W0, _W1 = 0x9E3779B9, 0xBB67AE85
_MASK = np.uint64(0xFFFFFFFF)


def philox4x32_10(ctr: np.ndarray, key: tuple[int, int]) -> np.ndarray:
    """Philox4x32 with 10 rounds.  ctr uint32 [..., 4]; returns uint32 [..., 4]."""
    c = [ctr[..., i].astype(np.uint64) for i in range(4)]
    k0, k1 = key[0] & 0xFFFFFFFF, key[1] & 0xFFFFFFFF
    for r in range(10):
        if r:
            k0 = (k0 + _W0) & 0xFFFFFFFF
            k1 = (k1 + _W1) & 0xFFFFFFFF
        p0 = _M0 * c[0]
        p1 = _M1 * c[2]
        c = [(p1 >> np.uint64(32)) ^ c[1] ^ np.uint64(k0), p1 & _MASK,
             (p0 >> np.uint64(32)) ^ c[3] ^ np.uint64(k1), p0 & _MASK]
    return np.stack([a.astype(np.uint32) for a in c], axis=-1)


def _f32(v: float) -> np.float32:
    return np.float32(v)


# ln 2 split into a high part with 8 trailing zero bits (so e * LN2_HI is exact
# for |e| < 256) and the float32 remainder.
_LN2_HI = np.array([math.log(2.0)], dtype=np.float32).view(np.uint32) & np.uint32(0xFFFFFF00)
_LN2_HI = _LN2_HI.view(np.float32)[0]
_LN2_LO = _f32(math.log(2.0) - float(_LN2_HI))
# 2*atanh(s)/s = sum_k 2 s^(2k) / (2k+1): Taylor coefficients, float32.
_C = [_f32(2.0 / (2 * k + 1)) for k in range(6)]
_SQRT2 = _f32(math.sqrt(2.0))


def own_log(x: np.ndarray) -> np.ndarray:
    """Natural log of positive normal float32 values, float32, fixed operation order.

    Method: x = 2^e m with m in [sqrt(1/2), sqrt(2)]; f = m - 1 (exact);
    s = f / (2 + f); ln m = 2 atanh(s) = s (C0 + z (C1 + z (C2 + ... ))) with
    z = s^2 and C_k = 2/(2k+1); ln x = e LN2_HI + (e LN2_LO + ln m).  Each
    product and sum is rounded to float32 separately.
    """
    x = np.asarray(x, dtype=np.float32)
    bits = x.view(np.uint32)
    e = ((bits >> np.uint32(23)).astype(np.int32) & 0xFF) - 127
    m = ((bits & np.uint32(0x7FFFFF)) | np.uint32(0x3F800000)).view(np.float32)
    big = m > _SQRT2
    m = np.where(big, m * _f32(0.5), m)
    e = np.where(big, e + 1, e)
    f = m - _f32(1.0)
    t = _f32(2.0) + f
    s = f / t
    z = s * s
    p = np.full_like(s, _C[5])
    for c in (_C[4], _C[3], _C[2], _C[1], _C[0]):
        p = p * z
        p = p + c
    lm = s * p
    ef = e.astype(np.float32)
    lo = ef * _LN2_LO
    lo = lo + lm
    hi = ef * _LN2_HI
    return hi + lo


def uniform_from_bits(x: np.ndarray) -> np.ndarray:
    """u = ((x >> 8) | 1) * 2^-24 as float32, in (0, 1)."""
    m = (np.asarray(x, dtype=np.uint32) >> np.uint32(8)) | np.uint32(1)
    return m.astype(np.float32) * _f32(2.0 ** -24)


def gumbel_from_bits(x: np.ndarray) -> np.ndarray:
    u = uniform_from_bits(x)
    return -own_log(-own_log(u))


def noise(seed: int, seq_uid: int, step: int, vocab: int) -> np.ndarray:
    """Standard Gumbel noise g_v, v < vocab, float32 [vocab]."""
    n4 = (vocab + 3) // 4
    ctr = np.zeros((n4, 4), dtype=np.uint32)
    ctr[:, 0] = np.arange(n4, dtype=np.uint32)
    ctr[:, 1] = np.uint32(step & 0xFFFFFFFF)
    ctr[:, 2] = np.uint32(seq_uid & 0xFFFFFFFF)
    x = philox4x32_10(ctr, (seed & 0xFFFFFFFF, (seed >> 32) & 0xFFFFFFFF)).reshape(-1)[:vocab]
    return gumbel_from_bits(x)


def argmax_lowest(s: np.ndarray, valid: np.ndarray) -> int:
    """Index of the largest s among valid entries, smallest index on ties; -1 if none valid."""
    if not valid.any():
        return -1
    best = np.max(s[valid])
    return int(np.flatnonzero(valid & (s == best))[0])


def sample_row(logits: np.ndarray, seq_uid: int, step: int, temperature: float, seed: int):
    """Draw one token from softmax(logits / T).  Returns (token, logprob float64)."""
    l = np.asarray(logits, dtype=np.float32)
    V = l.shape[0]
    T = _f32(temperature)
    sc = l if T == _f32(1.0) else l / T
    s = sc + noise(seed, seq_uid, step, V)
    valid = np.isfinite(l)
    tok = argmax_lowest(s, valid)
    if tok < 0:
        return -1, float("nan")
    z = l[valid].astype(np.float64) / float(T)
    m = z.max()
    lse = m + math.log(np.exp(z - m).sum())
    return tok, float(l[tok]) / float(T) - lse


def sample(logits: np.ndarray, seq_uid, step, temperature: float, seed: int, row_of=None):
    """Sample every row b from logits[row_of[b]] (or logits[b]).  Returns (int32 [B], float64 [B])."""
    seq_uid = np.asarray(seq_uid)
    step = np.broadcast_to(np.asarray(step), seq_uid.shape)
    B = seq_uid.shape[0]
    toks = np.empty(B, dtype=np.int32)
    lps = np.empty(B, dtype=np.float64)
    for b in range(B):
        r = b if row_of is None else int(row_of[b])
        toks[b], lps[b] = sample_row(logits[r], int(seq_uid[b]), int(step[b]), temperature, seed)
    return toks, lps
