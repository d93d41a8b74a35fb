"""bfloat16 rounding for the oracle (test infrastructure only).

bfloat16 keeps the top 16 bits of an IEEE binary32 value.  Conversion rounds
to nearest with ties to even on the 16 dropped bits.  NaN/Inf are not handled
(the workloads never produce them).
"""
import numpy as np


def round_bits(x) -> np.ndarray:
    """fp32 values -> uint16 bfloat16 bit patterns, round to nearest even."""
    b = np.ascontiguousarray(np.asarray(x, dtype=np.float32)).view(np.uint32).astype(np.uint64)
    lsb = (b >> np.uint64(16)) & np.uint64(1)
    r = (b + np.uint64(0x7FFF) + lsb) >> np.uint64(16)
    return (r & np.uint64(0xFFFF)).astype(np.uint16)


def bits_to_f32(h) -> np.ndarray:
    """uint16 bfloat16 bit patterns -> exact fp32 values."""
    h = np.asarray(h, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return h.view(np.float32)


def round_f32(x) -> np.ndarray:
    """fp32 values rounded to the nearest bfloat16, returned as fp32."""
    return bits_to_f32(round_bits(x))
