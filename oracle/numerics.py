"""bfloat16 helpers for the oracle (own implementation; shares nothing with the GPU path).

bfloat16 keeps the top 16 bits of an IEEE float32.  Rounding float32 to
bfloat16 is round-to-nearest, ties-to-even on the dropped 16 bits.  The
oracle computes in float64; ``round_bf16`` first rounds to float32 (nearest
even) and then to bfloat16, which is the order the GPU kernels use when
they store an fp32 accumulator as bf16.
"""
from __future__ import annotations

import numpy as np


def decode(arr: np.ndarray, dtype: str) -> np.ndarray:
    """Stored weights -> float64 (exact).  ``bf16`` arrays hold uint16 bit patterns."""
    if dtype == "bf16":
        bits = np.asarray(arr, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
        return bits.view(np.float32).astype(np.float64)
    return np.asarray(arr, dtype=np.float32).astype(np.float64)


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round float64 values to the nearest bfloat16 value (via float32), returned as float64."""
    f = np.asarray(x, dtype=np.float64).astype(np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    keep = u >> np.uint64(16)
    rem = u & np.uint64(0xFFFF)
    up = (rem > 0x8000) | ((rem == 0x8000) & ((keep & np.uint64(1)) == 1))
    keep = keep + up.astype(np.uint64)
    out = (keep.astype(np.uint32) << np.uint32(16)).view(np.float32)
    return out.astype(np.float64)


class Precision:
    """Where values are quantised.  ``bf16=False`` is the float32-config path (no rounding)."""

    def __init__(self, bf16: bool):
        self.bf16 = bf16

    def q(self, x: np.ndarray) -> np.ndarray:
        return round_bf16(x) if self.bf16 else x
