"""bf16 bit patterns -> fp64, exactly (test infrastructure; see oracle/__init__.py).

A bf16 value is the upper 16 bits of an IEEE-754 binary32 value, so placing the
pattern in the high half of a 32-bit word and reading it as binary32 recovers it
exactly; binary32 -> binary64 is exact as well.
"""
import numpy as np


def to_f64(bits: np.ndarray) -> np.ndarray:
    bits = np.asarray(bits)
    assert bits.dtype == np.uint16, bits.dtype
    return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
