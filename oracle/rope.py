"""Rotary position embedding, RMS normalisation of Q/K heads and the rotated
KV store -- TEST INFRASTRUCTURE ONLY (same rules as the rest of ``oracle/``).

Prefill materialises every suffix token's K/V before attention (paper,
Section 2).  The paper does not describe the layers that produce Q and K; the
models it serves (Qwen3, Section 4) normalise each Q and K head with an RMS norm
and then apply a rotary position embedding before K enters the cache.  This
module writes those steps out in float64 so that a fused "norm + rotate +
quantise + store" can be checked.  Readings (the paper is silent on all of them):

  * Position.  Suffix token i of a request with a cached prefix of P tokens sits
    at absolute position P + i of the request's logical sequence; its Q and K
    rotate by that position.
  * Rotation (RoFormer, Su et al., Section 3.2): the first ``rotary_dim`` dims of
    a head form rotary_dim/2 planes; plane j at position p turns by the angle
    p * f_j with f_j = theta^(-2j/rotary_dim) (or caller-given frequencies).
    Dims past rotary_dim pass through.  Plane j holds dims (j, j + rotary_dim/2)
    in the "half" layout (GPT-NeoX / Llama / Qwen) and dims (2j, 2j + 1) in the
    "interleaved" layout (GPT-J).  The turn maps (a, b) to
    (a cos - b sin, a sin + b cos).
  * RMS norm (when a weight is given): y = x * w / sqrt(mean(x^2) + eps) over
    all head_dim dims of one head, applied before the rotation.
  * Rounding: everything is exact real arithmetic here (float64); the result
    is rounded once -- to bf16 for Q and a bf16 pool, or to float32 and then
    encode(float32(x) * float32(1/scale)) for an fp8 pool (the store's reading).
"""

from __future__ import annotations

import numpy as np

from . import OraclePool, bf16_round, bf16_value, store_kv_values

HALF = 0
INTERLEAVED = 1

# Planted mistakes for the tests that show the checks tell a wrong rotation from
# the right one (never used by the oracle itself).
MUTANTS = ("none", "sin_sign", "position_plus_one", "freq_over_head_dim", "other_layout", "norm_after_rope")


def frequencies(theta: float, rotary_dim: int) -> np.ndarray:
    """f_j = theta^(-2j / rotary_dim), j = 0 .. rotary_dim/2 - 1 (RoFormer, Section 3.2.2)."""
    j = np.arange(rotary_dim // 2, dtype=np.float64)
    return np.power(np.float64(theta), -2.0 * j / rotary_dim)


def planes(rotary_dim: int, style: int):
    """Dim indices (first, second) of each rotation plane."""
    half = rotary_dim // 2
    j = np.arange(half)
    if style == HALF:
        return j, j + half
    if style == INTERLEAVED:
        return 2 * j, 2 * j + 1
    raise ValueError(f"style {style}")


def rope(x: np.ndarray, pos: np.ndarray, theta: float, rotary_dim: int, style: int = HALF,
         freqs=None, mutant: str = "none") -> np.ndarray:
    """Rotate x [n, H, d] (float64) by the positions pos [n]."""
    x = np.asarray(x, dtype=np.float64)
    d = x.shape[-1]
    if rotary_dim % 2 or not 0 < rotary_dim <= d:
        raise ValueError("rotary_dim must be even and in (0, head_dim]")
    if freqs is None:
        freqs = frequencies(theta, rotary_dim)
        if mutant == "freq_over_head_dim":
            freqs = frequencies(theta, d)[: rotary_dim // 2]
    freqs = np.asarray(freqs, dtype=np.float64)
    if freqs.shape != (rotary_dim // 2,):
        raise ValueError("need rotary_dim/2 frequencies")
    p = np.asarray(pos, dtype=np.float64) + (1 if mutant == "position_plus_one" else 0)
    ang = p[:, None] * freqs[None, :]                # [n, planes]
    c = np.cos(ang)[:, None, :]
    s = np.sin(ang)[:, None, :]
    if mutant == "sin_sign":
        s = -s
    first, second = planes(rotary_dim, INTERLEAVED if (mutant == "other_layout") != (style == INTERLEAVED)
                           else HALF)
    a = x[..., first]
    b = x[..., second]
    y = x.copy()
    y[..., first] = a * c - b * s
    y[..., second] = a * s + b * c
    return y


def rms_norm(x: np.ndarray, w, eps: float) -> np.ndarray:
    """y = x * w / sqrt(mean(x^2) + eps) over the last axis."""
    x = np.asarray(x, dtype=np.float64)
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * np.asarray(w, dtype=np.float64)


def positions(prefix_lens, extend_lens) -> np.ndarray:
    """Absolute position P_r + i of every suffix row, in row order."""
    out = [np.arange(p, p + e, dtype=np.int64) for p, e in zip(prefix_lens, extend_lens)]
    return np.concatenate(out) if out else np.zeros(0, np.int64)


def transform(bits, pos, theta, rotary_dim, style=HALF, norm_w=None, eps=1e-6, freqs=None,
              mutant="none") -> np.ndarray:
    """Exact values of the normalised, rotated heads of bf16 rows bits [n, H, d]."""
    x = bf16_value(bits)
    w = None if norm_w is None else bf16_value(norm_w)
    if mutant == "norm_after_rope":
        y = rope(x, pos, theta, rotary_dim, style, freqs)
        return y if w is None else rms_norm(y, w, eps)
    if w is not None:
        x = rms_norm(x, w, eps)
    return rope(x, pos, theta, rotary_dim, style, freqs, mutant)


def rotate_q(q_bits, prefix_lens, extend_lens, theta, rotary_dim, style=HALF, q_norm=None, eps=1e-6,
             freqs=None, mutant="none"):
    """(exact float64 values, nearest bf16 bits) of the rotated queries [T, Hq, d]."""
    pos = positions(prefix_lens, extend_lens)
    y = transform(q_bits, pos, theta, rotary_dim, style, q_norm, eps, freqs, mutant)
    return y, bf16_round(y)


def store_kv_rope(pool: OraclePool, prefix_lens, extend_lens, page_indptr, page_ids, k_bits, v_bits,
                  theta, rotary_dim, style=HALF, k_norm=None, eps=1e-6, freqs=None, mutant="none"):
    """Normalise and rotate the suffix keys, then store K and V into the pool.
    Returns the exact rotated keys (float64 [T, Hkv, d])."""
    pos = positions(prefix_lens, extend_lens)
    k = transform(k_bits, pos, theta, rotary_dim, style, k_norm, eps, freqs, mutant)
    store_kv_values(pool, prefix_lens, extend_lens, page_indptr, page_ids, k, v_bits)
    return k
