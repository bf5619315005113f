"""Rounding and activation helpers of the oracle (float64 NumPy).

Test infrastructure only; see the package docstring.

bf16 is IEEE binary32 truncated to 8 significant bits (1 implicit + 7
stored) with binary32's exponent range.  Rounding here is written out from
that definition: scale the value so that one unit in the last bf16 place
is 1, round half to even (``np.rint``), scale back.
"""
from __future__ import annotations

import numpy as np

_BF16_MAX = float(np.ldexp(255.0 / 128.0, 127))  # (2 - 2^-7) * 2^127


def round_bf16(a) -> np.ndarray:
    """Round float64 values to the nearest bf16 value, ties to even.

    Returns float64 holding bf16-representable values.  Subnormal bf16
    spacing (2^-133) is respected; values past the largest finite bf16
    round to +-inf when they are at or beyond the halfway point to 2^128.
    """
    a = np.asarray(a, dtype=np.float64)
    out = np.array(a, copy=True)
    finite = np.isfinite(a) & (a != 0.0)
    v = a[finite]
    _, e = np.frexp(v)                    # v = m * 2^e, 0.5 <= |m| < 1
    e = np.maximum(e, -125)               # below 2^-126 the spacing is fixed
    ulp_exp = e - 8                       # 8 significant bits
    r = np.ldexp(np.rint(np.ldexp(v, -ulp_exp)), ulp_exp)
    r = np.where(np.abs(r) > _BF16_MAX, np.copysign(np.inf, r), r)
    out[finite] = r
    return out


def round_f32(a) -> np.ndarray:
    """Round float64 values to float32 (IEEE RNE) and widen back."""
    return np.asarray(a, dtype=np.float64).astype(np.float32).astype(np.float64)


def rounder(dtype: str):
    """The rounding applied at the layer's rounding points for ``dtype``.

    "bf16" -> round_bf16, "f32" -> round_f32, "f64" -> identity (used by the
    finite-difference pins, where rounding would break differentiability).
    """
    if dtype == "bf16":
        return round_bf16
    if dtype == "f32":
        return round_f32
    if dtype == "f64":
        return lambda a: np.asarray(a, dtype=np.float64)
    raise ValueError(f"unknown dtype {dtype!r}")


def sigmoid(a) -> np.ndarray:
    a = np.asarray(a, dtype=np.float64)
    return 1.0 / (1.0 + np.exp(-a))


def silu(a) -> np.ndarray:
    """SiLU(a) = a * sigmoid(a) = a / (1 + e^-a)."""
    a = np.asarray(a, dtype=np.float64)
    return a / (1.0 + np.exp(-a))
