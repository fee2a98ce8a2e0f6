"""Elementary numerics of the oracle: storage rounding and the scalar functions
the method uses.  Test infrastructure only (see the package docstring).

Everything here works on float64 NumPy arrays.
"""
from __future__ import annotations

import numpy as np

# bf16 keeps the top 16 bits of an IEEE binary32: 1 sign, 8 exponent, 7 mantissa
# bits.  In binary64 terms that is 7 of the 52 stored mantissa bits, so rounding
# drops the low 45 bits.
_DROP = 45
_HALF_MINUS_ONE = np.uint64((1 << (_DROP - 1)) - 1)
_KEEP_MASK = np.uint64(~((1 << _DROP) - 1) & 0xFFFFFFFFFFFFFFFF)


def decode_bf16(bits: np.ndarray) -> np.ndarray:
    """uint16 bf16 bit patterns -> float64 values (exact)."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32)
    b <<= np.uint32(16)                      # in place: one temporary, not two
    return b.view(np.float32).astype(np.float64)


def as_f64(x: np.ndarray) -> np.ndarray:
    """Input tensor (uint16 bf16 bits, float32 or float64) -> float64 values."""
    x = np.asarray(x)
    if x.dtype == np.uint16:
        return decode_bf16(x)
    return x.astype(np.float64, copy=False)


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round float64 values to the nearest bf16 value, ties to even, returned as
    float64.  Done directly on the binary64 encoding (one rounding, no detour
    through binary32).  Values must be finite and at least 2^-126 in magnitude
    or zero (bf16 normal range); smaller magnitudes are flushed to signed zero,
    which no workload here produces."""
    x = np.ascontiguousarray(np.asarray(x, dtype=np.float64))
    u = x.view(np.uint64)
    lsb = (u >> np.uint64(_DROP)) & np.uint64(1)
    r = ((u + _HALF_MINUS_ONE + lsb) & _KEEP_MASK).view(np.float64)
    tiny = np.abs(r) < 2.0 ** -126
    if np.any(tiny):
        r = np.where(tiny, np.copysign(0.0, x), r)
    return r


def encode_bf16(x: np.ndarray) -> np.ndarray:
    """float64 values that are exactly bf16 -> uint16 bit patterns."""
    f = np.asarray(x, dtype=np.float64).astype(np.float32)
    return (f.view(np.uint32) >> np.uint32(16)).astype(np.uint16)


def round_f32(x: np.ndarray) -> np.ndarray:
    """Round to the nearest binary32 (ties to even), returned as float64."""
    return np.asarray(x, dtype=np.float64).astype(np.float32).astype(np.float64)


def store(x: np.ndarray, dtype: str) -> np.ndarray:
    """Storage rounding of a tensor that the GPU path keeps in ``dtype``."""
    if dtype == "bf16":
        return round_bf16(x)
    if dtype == "f32":
        return round_f32(x)
    raise ValueError(dtype)


def sigmoid(z: np.ndarray) -> np.ndarray:
    """Logistic function 1 / (1 + e^{-z}), the per-path gate of Eq. (1)."""
    z = np.asarray(z, dtype=np.float64)
    with np.errstate(over="ignore"):
        return 1.0 / (1.0 + np.exp(-z))


def silu(x: np.ndarray) -> np.ndarray:
    """SiLU(x) = x * sigmoid(x), the activation of the drafter's gated MLP."""
    return x * sigmoid(x)


def rmsnorm(x: np.ndarray, gamma, eps: float) -> np.ndarray:
    """RMSNorm over the last axis: x / sqrt(mean(x^2) + eps) * gamma."""
    x = np.asarray(x, dtype=np.float64)
    ms = np.mean(x * x, axis=-1, keepdims=True)
    y = x / np.sqrt(ms + eps)
    if gamma is not None:
        y = y * np.asarray(gamma, dtype=np.float64)
    return y
