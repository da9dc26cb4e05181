"""Exact bf16 -> fp64 decode (test infrastructure only).

A bf16 value is the upper 16 bits of an IEEE-754 binary32, so widening the
pattern by 16 zero bits gives the binary32 value exactly, and binary32 ->
binary64 is exact as well.
"""
import numpy as np


def to_f64(bits: np.ndarray) -> np.ndarray:
    """uint16 bf16 patterns -> float64 (exact)."""
    b = np.asarray(bits)
    if b.dtype != np.uint16:
        raise TypeError("expected uint16 bf16 bit patterns")
    return (b.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def from_f64_rne(x: np.ndarray) -> np.ndarray:
    """float64 -> nearest bf16 (ties to even), computed from the binary64 value.

    Used only where the checker must take a rounding decision in bf16.  Works
    on the exact binary64 value: finds the two neighbouring bf16 numbers by
    truncating the binary32 pattern and picks the nearer one.
    """
    x = np.asarray(x, dtype=np.float64)
    f = x.astype(np.float32)  # RNE to binary32 first cannot create a tie at bf16
    # f may differ from x; resolve with exact comparison on the two candidates.
    u = f.view(np.uint32)
    lo = (u & np.uint32(0xFFFF0000))
    hi = lo + np.uint32(0x10000)
    lo_v = lo.view(np.float32).astype(np.float64)
    hi_v = hi.view(np.float32).astype(np.float64)
    dlo = np.abs(x - lo_v)
    dhi = np.abs(hi_v - x)
    even_lo = ((lo >> 16) & 1) == 0
    pick_hi = (dhi < dlo) | ((dhi == dlo) & ~even_lo)
    out = np.where(pick_hi, hi, lo) >> 16
    return out.astype(np.uint16)
