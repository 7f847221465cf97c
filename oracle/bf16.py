"""bfloat16 rounding used by the oracle's bf16 precision recipe.

``round_bf16`` maps a float64/float32 array to the nearest bfloat16 value
(ties to even) by way of float32: first IEEE rounding to float32, then
round-to-nearest-even on the upper 16 bits.  The result is returned as
float64 (bf16 values are exact in float64).  Pinned against torch's own
float32 -> bfloat16 conversion in the CPU tests.
"""
from __future__ import annotations

import numpy as np


def round_bf16(x) -> np.ndarray:
    f = np.ascontiguousarray(np.asarray(x, dtype=np.float32))
    if not np.all(np.isfinite(f)):
        raise ValueError("round_bf16: non-finite input")
    b = f.view(np.uint32).astype(np.uint64)
    r = ((b + 0x7FFF + ((b >> 16) & 1)) >> 16) << 16
    return r.astype(np.uint32).view(np.float32).astype(np.float64)


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """uint16 bf16 bit patterns -> float64 values."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return b.view(np.float32).astype(np.float64)
