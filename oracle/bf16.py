"""bfloat16 <-> fp32 conversion for the oracle (test infrastructure only).

A bf16 value is the upper 16 bits of an IEEE binary32 value.  Widening is
exact (shift left by 16).  Narrowing rounds to nearest, ties to even, on the
16 discarded bits; NaNs stay NaN (quiet bit forced).  Written from the
definition of the format, not from any library routine.
"""

import numpy as np


def bf16_to_f32(u16):
    """uint16 array of bf16 bit patterns -> float32 array (exact)."""
    u16 = np.asarray(u16, dtype=np.uint16)
    return (u16.astype(np.uint32) << np.uint32(16)).view(np.float32)


def f32_to_bf16(f32):
    """float32 array -> uint16 bf16 bit patterns, round to nearest even."""
    f = np.ascontiguousarray(f32, dtype=np.float32)
    u = f.view(np.uint32).astype(np.uint64)          # no wrap on the add
    lsb = (u >> np.uint64(16)) & np.uint64(1)        # ties go to even
    r = ((u + np.uint64(0x7FFF) + lsb) >> np.uint64(16)).astype(np.uint16)
    nan = np.isnan(f)
    if nan.any():
        r[nan] = ((f.view(np.uint32)[nan] >> np.uint32(16))
                  | np.uint32(0x0040)).astype(np.uint16)
    return r
