"""Oracle for FP8 scaled quantization (paper Sec. 2.2, Eq. 3) and the exact
scaled FP8 GEMM of the linear layer.

TEST INFRASTRUCTURE ONLY.  Plain, slow, single-threaded C compiled with gcc
(``liboracle.so``), wrapped here with ctypes and numpy.  Only ``tests/``,
``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py`` may
import this package.  It shares no code with the HIP library and the HIP
library never calls it.

Readings of the paper fixed by the oracle are documented in ``oracle.h``.
"""
import ctypes
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(HERE, "liboracle.so")
SOURCES = ["e4m3.c", "e5m2.c", "quantize.c", "gemm.c"]

TENSOR, ROW, COL, BLOCK_1x128, BLOCK_128x1, BLOCK_128x128 = range(6)
OUT_TRANSPOSED = 1
POW2_SCALE = 2
E5M2 = 4                    # quantize flag: E5M2 codes, F_max = 57344
FMT_E4M3, FMT_E5M2 = 0, 1   # GEMM operand formats


def build(force=True):
    """Compile liboracle.so with gcc: no fast-math, no FMA contraction."""
    if not force and os.path.exists(LIB):
        return LIB
    srcs = [os.path.join(HERE, s) for s in SOURCES]
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = ["gcc", "-std=c11", "-O2", "-ffp-contract=off", "-fno-fast-math",
           "-fPIC", "-shared", "-Wall", "-Wextra", "-o", tmp] + srcs + ["-lm"]
    subprocess.check_call(cmd)
    os.replace(tmp, LIB)
    return LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB):
            build()
        L = ctypes.CDLL(LIB)
        p, i64, i32, u32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_uint
        L.oracle_e4m3_decode.argtypes = [ctypes.c_uint8]
        L.oracle_e4m3_decode.restype = ctypes.c_double
        L.oracle_e4m3_encode.argtypes = [ctypes.c_float]
        L.oracle_e4m3_encode.restype = ctypes.c_uint8
        L.oracle_cast_f32.argtypes = [ctypes.c_float, ctypes.c_float]
        L.oracle_cast_f32.restype = ctypes.c_uint8
        L.oracle_cast_f32_array.argtypes = [p, i64, ctypes.c_float, p]
        L.oracle_cast_f32_array.restype = None
        L.oracle_e5m2_decode.argtypes = [ctypes.c_uint8]
        L.oracle_e5m2_decode.restype = ctypes.c_double
        L.oracle_e5m2_encode.argtypes = [ctypes.c_float]
        L.oracle_e5m2_encode.restype = ctypes.c_uint8
        L.oracle_cast_f32_e5m2_array.argtypes = [p, i64, ctypes.c_float, p]
        L.oracle_cast_f32_e5m2_array.restype = None
        L.oracle_quantize.argtypes = [p, i64, i64, i64, i32, u32, p, i64, p]
        L.oracle_quantize.restype = i32
        L.oracle_gemm_rows.argtypes = [p, p, i32, i64, p, p, i32, i64,
                                       i64, i64, i64, p, i64, p]
        L.oracle_gemm_rows.restype = i32
        L.oracle_gemm_rows_fmt.argtypes = [p, p, i32, i64, i32, p, p, i32, i64, i32,
                                           i64, i64, i64, p, i64, p]
        L.oracle_gemm_rows_fmt.restype = i32
        _lib = L
    return _lib


def _ptr(a):
    return a.ctypes.data_as(ctypes.c_void_p)


def decode(code):
    return lib().oracle_e4m3_decode(int(code))


def encode(v):
    return lib().oracle_e4m3_encode(float(v))


def decode_e5m2(code):
    return lib().oracle_e5m2_decode(int(code))


def encode_e5m2(v):
    return lib().oracle_e5m2_encode(float(v))


def cast_f32(x, scale, e5m2=False):
    """Q_FP8(RN32(x / scale)) elementwise (E4M3, or E5M2); x is a float32 array."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    out = np.empty(x.shape, dtype=np.uint8)
    fn = lib().oracle_cast_f32_e5m2_array if e5m2 else lib().oracle_cast_f32_array
    fn(_ptr(x), x.size, float(scale), _ptr(out))
    return out


def scale_count(rows, cols, granularity):
    return {TENSOR: 1, ROW: rows, COL: cols,
            BLOCK_1x128: rows * (cols // 128), BLOCK_128x1: (rows // 128) * cols,
            BLOCK_128x128: (rows // 128) * (cols // 128)}[granularity]


def quantize(x_bits, granularity, transposed=False, pow2=False, e5m2=False):
    """Eq. 3 per scaling unit (pow2: the power-of-two scale variant; e5m2:
    E5M2 codes with F_max = 57344).

    x_bits: uint16 array [rows, cols] of bf16 bit patterns.
    Returns (codes uint8 [rows, cols] or [cols, rows], scales float32 1-D).
    """
    x_bits = np.ascontiguousarray(x_bits, dtype=np.uint16)
    rows, cols = x_bits.shape
    orows, ocols = (cols, rows) if transposed else (rows, cols)
    og = granularity
    if transposed:
        og = {ROW: COL, COL: ROW, BLOCK_1x128: BLOCK_128x1,
              BLOCK_128x1: BLOCK_1x128}.get(granularity, granularity)
    codes = np.empty((orows, ocols), dtype=np.uint8)
    scales = np.empty(scale_count(orows, ocols, og), dtype=np.float32)
    rc = lib().oracle_quantize(_ptr(x_bits), rows, cols, cols, granularity,
                               (OUT_TRANSPOSED if transposed else 0) | (POW2_SCALE if pow2 else 0)
                               | (E5M2 if e5m2 else 0),
                               _ptr(codes), ocols, _ptr(scales))
    if rc != 0:
        raise ValueError("oracle_quantize rejected the arguments")
    return codes, scales


def gemm_rows(A, sA, gA, B, sB, gB, rows, fmtA=FMT_E4M3, fmtB=FMT_E4M3):
    """Exact C[rows, :] of the scaled FP8 GEMM, fp64.

    A: uint8 [M, K] codes, B: uint8 [N, K] codes (K contiguous), each in
    E4M3 or E5M2 (FMT_*).
    """
    A = np.ascontiguousarray(A, dtype=np.uint8)
    B = np.ascontiguousarray(B, dtype=np.uint8)
    sA = np.ascontiguousarray(sA, dtype=np.float32)
    sB = np.ascontiguousarray(sB, dtype=np.float32)
    rows = np.ascontiguousarray(rows, dtype=np.int64)
    M, K = A.shape
    N, K2 = B.shape
    assert K == K2
    out = np.empty((rows.size, N), dtype=np.float64)
    rc = lib().oracle_gemm_rows_fmt(_ptr(A), _ptr(sA), gA, K, fmtA, _ptr(B), _ptr(sB),
                                    gB, K, fmtB, M, N, K, _ptr(rows), rows.size,
                                    _ptr(out))
    if rc != 0:
        raise ValueError("oracle_gemm_rows rejected the arguments")
    return out
