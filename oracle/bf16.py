"""Exact widening of bfloat16 bit patterns to float64 (oracle side).

A bfloat16 value is the upper 16 bits of an IEEE-754 binary32 value, so
shifting the pattern left by 16 bits gives the binary32 value exactly, and
binary32 -> binary64 is exact.  Test infrastructure only.
"""
import numpy as np


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    bits = np.asarray(bits, dtype=np.uint16)
    return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)
