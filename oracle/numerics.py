"""Rounding points of the oracle.

bfloat16 keeps the top 16 bits of an IEEE-754 binary32 value.  Rounding a
binary32 value to bfloat16 "to nearest, ties to even" adds 0x7FFF plus the
lowest kept bit to the bit pattern and truncates the low 16 bits; a carry into
the exponent rounds up to the next binade (or to infinity), which is exactly
round-to-nearest-even.  NaNs stay NaN.
"""
import numpy as np


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """uint16 bfloat16 bit patterns -> float32 values (exact)."""
    return (np.asarray(bits).astype(np.uint32) << np.uint32(16)).view(np.float32)


def rne_bf16(x) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even); returns
    float32 arrays holding bfloat16-representable values."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    r = ((u + np.uint64(0x7FFF) + lsb) >> np.uint64(16)) << np.uint64(16)
    out = r.astype(np.uint32).view(np.float32).copy()
    nan = np.isnan(x)
    if nan.any():
        out[nan] = np.float32(np.nan)
    return out.reshape(x.shape)


def to_f32(x64: np.ndarray) -> np.ndarray:
    """float64 -> float32, round to nearest even (IEEE conversion)."""
    return np.asarray(x64, dtype=np.float64).astype(np.float32)
