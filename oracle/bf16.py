"""fp32 -> bfloat16 round-to-nearest-even, as plain integer arithmetic.

Test infrastructure (see the package docstring).  The paper names no numeric
precision; the library's bf16 path rounds GEMM inputs (x, W_x, W_h, W_p
and the hidden states fed back into the recurrence) to bfloat16.  The oracle
reference for that path takes the same rounded inputs and keeps everything
else in fp64.
"""
import numpy as np


def round_to_bf16(a):
    """Round an array to the nearest bfloat16 value (ties to even).

    The input is first taken to float32; the result is returned as float64
    holding exactly representable bfloat16 values.  NaN stays NaN.
    """
    f = np.ascontiguousarray(np.asarray(a, dtype=np.float32))
    u = f.view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    rounded = (u + 0x7FFF + lsb) >> 16
    out = (rounded << 16).astype(np.uint32).view(np.float32)
    out = np.where(np.isnan(f), np.float32(np.nan), out)
    return out.astype(np.float64)


def bf16_bits(a):
    """The 16-bit patterns of ``round_to_bf16(a)`` (uint16 array)."""
    r = round_to_bf16(a).astype(np.float32)
    return (r.view(np.uint32) >> 16).astype(np.uint16)
