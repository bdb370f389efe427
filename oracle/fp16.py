"""fp16 <-> fp64 conversions used throughout the oracle.

The quantizer stores its scale, zero and centroids as fp16 (Method, section 3.2:
packed scalar quantizers with exact scale overhead).  A value computed in fp64 is
stored with ONE round-to-nearest-even to fp16; it never passes through fp32 on
the way (that would round twice).  numpy's float64 -> float16 cast rounds
directly; ``tests/test_oracle_fp16_ladder.py`` pins that with vectors where a detour
through fp32 gives a different answer.

Zero is canonicalised to +0 wherever the oracle stores a value that is compared
bit for bit (boxes, scales, zeros, centroids), so the sign of a zero never
decides parity.
"""
import numpy as np


def to_f64(bits):
    """fp16 bit patterns (uint16 array) -> exact float64 values."""
    return np.asarray(bits, dtype=np.uint16).view(np.float16).astype(np.float64)


def from_f64(x):
    """float64 values -> fp16 bit patterns with a single RNE rounding; -0 -> +0."""
    h = np.asarray(x, dtype=np.float64).astype(np.float16)
    bits = h.view(np.uint16).copy()
    bits[bits == 0x8000] = 0
    return bits


def canon_zero_bits(bits):
    """Map the fp16 pattern of -0 to +0 (other patterns unchanged)."""
    b = np.asarray(bits, dtype=np.uint16).copy()
    b[b == 0x8000] = 0
    return b
