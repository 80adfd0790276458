"""The quantizer kernels form RN32(x / S) from the reciprocal of S with one
residual correction instead of a division per element.  This CPU test checks
that sequence over every (bf16 amax, bf16 x) pair the kernels can meet,
signs and signed zeros included, against the correctly rounded quotient:
the E4M3 codes (and, for the E5M2 variant, the E5M2 codes) must never
differ.  (The GPU tests then compare the kernels with the oracle on the
same exhaustive set.)"""
import ctypes
import os

import pytest

from _cbuild import helper


@pytest.mark.parametrize("e5m2", [0, 1], ids=["e4m3", "e5m2"])
def test_quotient_sequence_exhaustive(e5m2):
    """E4M3 with F_max = 448, and the E5M2 variant with F_max = 57344."""
    lib = helper("div_sweep")
    lib.div_sweep_fmt.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.POINTER(ctypes.c_uint64),
                                  ctypes.POINTER(ctypes.c_uint32), ctypes.POINTER(ctypes.c_uint32)]
    lib.div_sweep_fmt.restype = ctypes.c_uint64
    pairs, a, x = ctypes.c_uint64(), ctypes.c_uint32(), ctypes.c_uint32()
    threads = min(16, len(os.sched_getaffinity(0)))
    bad = lib.div_sweep_fmt(threads, e5m2, ctypes.byref(pairs), ctypes.byref(a), ctypes.byref(x))
    # sum over amax a of (a + 1) magnitudes, two signs each
    assert pairs.value == 2 * sum(a_ + 1 for a_ in range(1, 0x7F80))
    assert bad == 0, "code differs for amax bits %#06x, x bits %#06x" % (a.value, x.value)
