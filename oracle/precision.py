"""Working precision of the oracle's floating-point arrays.

Test infrastructure (see the package docstring).  Every reference value the
tests compare against is computed in fp64, the default.  The CPU baseline of
the benchmark also times the same code with fp32 arrays (``working``), the
precision a plain CPU implementation of the method would use in practice.
"""
import contextlib

import numpy as np

_FLOAT = np.float64


def F():
    """The current floating-point array type (np.float64 unless ``working``)."""
    return _FLOAT


@contextlib.contextmanager
def working(dtype):
    """Run the enclosed oracle calls with arrays of ``dtype``."""
    global _FLOAT
    old = _FLOAT
    _FLOAT = np.dtype(dtype).type
    try:
        yield
    finally:
        _FLOAT = old
