"""Storage roundings used by the oracle (bf16 round-to-nearest-even).

The paper does not state a precision.  The build's reading: in bf16 mode every
tensor stored between kernels is bf16 (weights, activations, the projection
XU, the perturbed coefficients C +/- eps Z, layer outputs), every product is
accumulated in fp32 or wider, and each stored value is rounded once with
round-to-nearest-even.  The oracle emulates each rounding point with the bit
arithmetic below.  Pinned by tests/test_oracle_core.py (exhaustive agreement
with torch's bfloat16 cast on all fp32 bit patterns of one exponent range, and
ties-to-even cases).
"""
from __future__ import annotations

import numpy as np


def rne_bf16(x) -> np.ndarray:
    """Round float values to bf16 (nearest, ties to even); returns float32 holding bf16 values."""
    b = np.ascontiguousarray(np.asarray(x, dtype=np.float32)).view(np.uint32)
    lsb = (b >> np.uint32(16)) & np.uint32(1)
    r = (b + np.uint32(0x7FFF) + lsb) & np.uint32(0xFFFF0000)
    return r.view(np.float32)


def as_f32(x) -> np.ndarray:
    return np.asarray(x, dtype=np.float32)
