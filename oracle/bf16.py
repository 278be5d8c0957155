"""Oracle helper: exact widening of bf16 bit patterns to float64.

Test infrastructure only.  A bf16 value is the upper half of an IEEE-754 binary32
word, so shifting the 16-bit pattern left by 16 gives the float32 with the same value,
which float64 represents exactly.
"""
import numpy as np


def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    u = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return u.view(np.float32).astype(np.float64)
