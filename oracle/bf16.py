"""bfloat16 storage for the oracle (numpy has no bf16 type).

Test infrastructure (see the package docstring).  A bf16 value is the upper
16 bits of an IEEE binary32 value; it is held here as its uint16 bit pattern.
Widening is exact (shift into the high half).  Narrowing from binary32 rounds
to nearest, ties to even, on the integer bit pattern; NaN stays NaN (quiet
bit set), infinities and signed zeros pass through, overflow rounds to inf.
"""
from __future__ import annotations

import numpy as np


def to_f64(bits) -> np.ndarray:
    """uint16 bf16 patterns -> float64 (exact)."""
    u = np.asarray(bits).astype(np.uint32) << np.uint32(16)
    with np.errstate(invalid="ignore"):
        return u.view(np.float32).astype(np.float64)


def from_f32(x) -> np.ndarray:
    """binary32 values -> bf16 bit patterns, round to nearest even."""
    f = np.ascontiguousarray(np.asarray(x, dtype=np.float32))
    u = f.view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    rounded = (u + np.uint64(0x7FFF) + lsb) >> np.uint64(16)
    is_nan = np.isnan(f)
    nan_bits = (u >> np.uint64(16)) | np.uint64(0x0040)
    out = np.where(is_nan, nan_bits, rounded)
    return out.astype(np.uint16)
