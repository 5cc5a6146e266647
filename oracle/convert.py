"""Element-type conversion for the weight-synchronising reshard (test infrastructure; see package header).

Actor training and actor generation are separate model-stages whose weights are synchronised at safe
boundaries (paper section 5, EMU definition): the training stage holds fp32 state, the generation stage
bf16 weights, in another layout. The reshard between them therefore also converts the element type.
The paper does not state a rounding rule; the reading taken here is the IEEE-754 default:

* fp32 -> bf16: keep the top 16 bits after rounding the low 16 bits to nearest, ties to even; values
  beyond the largest bf16 round to infinity; infinities stay infinities; a NaN stays a NaN with its sign
  and top payload bits and the quiet bit set (so a signalling NaN never becomes infinity).
* bf16 -> fp32: exact (the bf16 bits become the top 16 bits).

Arrays hold bit patterns: bf16 as uint16, fp32 as float32 (read through a uint32 view).
"""
from __future__ import annotations

import numpy as np


def f32_to_bf16(x: np.ndarray) -> np.ndarray:
    """Round fp32 values (float32 array) to bf16 bit patterns (uint16), nearest-even."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    is_nan = (u & 0x7FFF_FFFF) > 0x7F80_0000
    lsb = (u >> 16) & 1
    rounded = (u + 0x7FFF + lsb) >> 16
    quiet = (u >> 16) | 0x0040
    return np.where(is_nan, quiet, rounded).astype(np.uint16)


def bf16_to_f32(b: np.ndarray) -> np.ndarray:
    """Widen bf16 bit patterns (uint16) to fp32 values, exactly."""
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def convert(x: np.ndarray, src: str, dst: str) -> np.ndarray:
    """Convert one array of element type ``src`` to ``dst`` (each "bf16" or "fp32")."""
    if src == dst:
        return np.array(x, copy=True)
    if (src, dst) == ("fp32", "bf16"):
        return f32_to_bf16(x)
    if (src, dst) == ("bf16", "fp32"):
        return bf16_to_f32(x)
    raise ValueError(f"unsupported conversion {src} -> {dst}")
