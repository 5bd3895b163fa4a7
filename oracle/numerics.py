"""Scalar building blocks of the CPU oracle, in float64.

Test infrastructure only: nothing in the product imports this package.

Every function here is the textbook definition of one operation of the
transformer forward, evaluated in float64; ``round_to`` models the storage
dtype of the workload (fp32, bfloat16 or fp16) at the points where the
program stores a tensor.
"""
from __future__ import annotations

import numpy as np
from scipy.special import erf

F32, BF16, F16 = "f32", "bf16", "f16"

_BF16_MIN_NORMAL = 2.0 ** -126
_BF16_MIN_SUB = 2.0 ** -133
_BF16_MAX = float.fromhex("0x1.fep127")


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round float64 values to the nearest bfloat16 value (ties to even),
    returned as float64.  Normal numbers keep 8 significant bits; values
    below the smallest normal are rounded to multiples of 2**-133; values
    whose rounded magnitude exceeds the largest finite bfloat16 become inf.
    NaN stays NaN."""
    x = np.asarray(x, dtype=np.float64)
    u = x.view(np.uint64) if x.flags.c_contiguous else np.ascontiguousarray(x).view(np.uint64)
    drop = np.uint64(45)                      # 52 - 7 mantissa bits dropped
    half = np.uint64((1 << 44) - 1)
    lsb = (u >> drop) & np.uint64(1)
    r = (u + half + lsb) & ~np.uint64((1 << 45) - 1)
    out = r.view(np.float64).reshape(x.shape)
    small = np.abs(x) < _BF16_MIN_NORMAL
    if small.any():
        out = np.where(small, np.round(x / _BF16_MIN_SUB) * _BF16_MIN_SUB, out)
    big = np.abs(out) > _BF16_MAX
    if big.any():
        out = np.where(big, np.copysign(np.inf, x), out)
    nan = np.isnan(x)
    if nan.any():
        out = np.where(nan, np.nan, out)
    return out


def round_to(x: np.ndarray, dtype: str) -> np.ndarray:
    """Value of ``x`` after it is stored in ``dtype`` (as float64)."""
    x = np.asarray(x, dtype=np.float64)
    if dtype == F32:
        return x.astype(np.float32).astype(np.float64)
    if dtype == BF16:
        return round_bf16(x)
    if dtype == F16:
        with np.errstate(over="ignore"):
            return x.astype(np.float16).astype(np.float64)
    raise ValueError(dtype)


def decode(a: np.ndarray, dtype: str) -> np.ndarray:
    """Storage array (float32 / bfloat16 bits in uint16 / float16) -> float64."""
    if dtype == BF16:
        assert a.dtype == np.uint16
        return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return np.asarray(a).astype(np.float64)


def to_storage(x: np.ndarray, dtype: str) -> np.ndarray:
    """float64 values already representable in ``dtype`` -> storage array."""
    if dtype == F32:
        return x.astype(np.float32)
    if dtype == F16:
        with np.errstate(over="ignore"):
            return x.astype(np.float16)
    f = x.astype(np.float32)          # exact: bf16 values are float32 values
    return (f.view(np.uint32) >> 16).astype(np.uint16)


def gelu(x: np.ndarray) -> np.ndarray:
    """GELU with the exact Gaussian CDF: x * Phi(x) = 0.5 x (1 + erf(x/sqrt2))."""
    return 0.5 * x * (1.0 + erf(x / np.sqrt(2.0)))


def silu(x: np.ndarray) -> np.ndarray:
    """SiLU: x * sigmoid(x), written so that large |x| does not overflow."""
    with np.errstate(over="ignore"):
        return x / (1.0 + np.exp(-x))


def layer_norm(x: np.ndarray, g: np.ndarray, b: np.ndarray, eps: float) -> np.ndarray:
    """Row-wise LayerNorm with the biased variance."""
    mu = x.mean(axis=-1, keepdims=True)
    xc = x - mu
    var = (xc * xc).mean(axis=-1, keepdims=True)
    return xc / np.sqrt(var + eps) * g + b


def rms_norm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    """Row-wise RMSNorm: x / sqrt(mean(x^2) + eps) * g."""
    ms = (x * x).mean(axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * g


def masked_softmax(s: np.ndarray, allowed: np.ndarray) -> np.ndarray:
    """Softmax over the last axis restricted to ``allowed`` entries; entries
    not allowed get weight exactly 0, and a row with no allowed entry is all
    zeros."""
    neg = np.where(allowed, s, -np.inf)
    m = neg.max(axis=-1, keepdims=True)
    m = np.where(np.isfinite(m), m, 0.0)
    e = np.where(allowed, np.exp(np.where(allowed, s, m) - m), 0.0)
    z = e.sum(axis=-1, keepdims=True)
    return np.where(z > 0, e / np.where(z > 0, z, 1.0), 0.0)


def rope_table(n_pos: int, head_dim: int, base: float):
    """cos/sin tables [n_pos, head_dim/2] for rotary position embedding.

    theta_i = base ** (-2 i / head_dim); angle = p * theta_i.  Both the
    frequencies and the table entries are rounded to float32 (the table is
    stored in float32); everything else is float64."""
    half = head_dim // 2
    i = np.arange(half, dtype=np.float64)
    theta = (base ** (-2.0 * i / head_dim)).astype(np.float32).astype(np.float64)
    ang = np.arange(n_pos, dtype=np.float64)[:, None] * theta[None, :]
    return (np.cos(ang).astype(np.float32).astype(np.float64),
            np.sin(ang).astype(np.float32).astype(np.float64))


def rope_table_scaled(n_pos: int, head_dim: int, base: float, factor: np.ndarray,
                      attn: float):
    """cos/sin tables [n_pos, head_dim/2] of a scaled rotary frequency set
    (the long/short factors of a long-context rope).

    theta_i = 1 / (factor_i * base ** (2 i / head_dim)), with the power
    rounded to float32 and the product and the quotient as float32
    operations (the frequency buffer is float32); angle = p * theta_i in
    float64; cos and sin rounded to float32 and multiplied by ``attn`` as a
    float32 product."""
    half = head_dim // 2
    i = np.arange(half, dtype=np.float64)
    ib = (base ** (2.0 * i / head_dim)).astype(np.float32)
    denom = (np.asarray(factor, dtype=np.float32) * ib).astype(np.float32)
    theta = (np.float32(1.0) / denom).astype(np.float32).astype(np.float64)
    ang = np.arange(n_pos, dtype=np.float64)[:, None] * theta[None, :]
    a = np.float32(attn)
    c = (np.cos(ang).astype(np.float32) * a).astype(np.float32)
    s = (np.sin(ang).astype(np.float32) * a).astype(np.float32)
    return c.astype(np.float64), s.astype(np.float64)


def apply_rope(x: np.ndarray, cos: np.ndarray, sin: np.ndarray) -> np.ndarray:
    """Rotate-half rotary embedding on the last axis (pairs i, i + hd/2).
    ``x`` is [..., S, hd]; ``cos``/``sin`` are [S, hd/2]."""
    half = x.shape[-1] // 2
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * cos - x2 * sin, x2 * cos + x1 * sin], axis=-1)
