"""Test-side helpers: the oracle run on row chunks in parallel threads (its
ctypes calls release the GIL; each chunk is a plain oracle call), and the
GEMM error measure."""
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

import oracle

THREADS = max(1, min(16, len(os.sched_getaffinity(0))))

_ROW_LOCAL = {oracle.BLOCK_1x128: 1, oracle.BLOCK_128x1: 128,
              oracle.BLOCK_128x128: 128, oracle.ROW: 1}


def quantize(x_bits, g, transposed=False, threads=THREADS, pow2=False, e5m2=False):
    """oracle.quantize on a [rows, cols] bf16 bit array, split into row chunks
    when the granularity's units do not cross rows of the chunking."""
    rows, cols = x_bits.shape
    step = _ROW_LOCAL.get(g)
    if step is None or rows <= 1024:
        return oracle.quantize(x_bits, g, transposed, pow2, e5m2)
    nchunk = min(threads * 4, rows // step)
    bounds = np.linspace(0, rows // step, nchunk + 1).astype(np.int64) * step
    bounds[-1] = rows
    parts = [(int(a), int(b)) for a, b in zip(bounds[:-1], bounds[1:]) if b > a]
    with ThreadPoolExecutor(threads) as ex:
        res = list(ex.map(lambda ab: oracle.quantize(x_bits[ab[0]:ab[1]], g, transposed, pow2, e5m2), parts))
    codes = np.concatenate([c for c, _ in res], axis=1 if transposed else 0)
    if g == oracle.BLOCK_1x128:       # [cols/128][rows], chunks along rows
        scales = np.concatenate([s.reshape(cols // 128, -1) for _, s in res], axis=1).reshape(-1)
    elif g == oracle.BLOCK_128x128 and transposed:  # [cols/128][rows/128]
        scales = np.concatenate([s.reshape(cols // 128, -1) for _, s in res], axis=1).reshape(-1)
    else:                             # row-major in the chunked dimension
        scales = np.concatenate([s for _, s in res])
    return codes, scales


def gemm_rows(A, sA, gA, B, sB, gB, rows, threads=THREADS, fmtA=oracle.FMT_E4M3, fmtB=oracle.FMT_E4M3):
    rows = np.asarray(rows, dtype=np.int64)
    parts = np.array_split(rows, max(1, min(threads * 2, rows.size)))
    with ThreadPoolExecutor(threads) as ex:
        res = list(ex.map(lambda r: oracle.gemm_rows(A, sA, gA, B, sB, gB, r, fmtA, fmtB), parts))
    return np.concatenate(res, axis=0)


def cast_f32(x, scale, threads=THREADS, e5m2=False):
    parts = np.array_split(x, threads * 4)
    with ThreadPoolExecutor(threads) as ex:
        res = list(ex.map(lambda p: oracle.cast_f32(p, scale, e5m2), parts))
    return np.concatenate(res)


def rel_err(got, ref):
    """Max relative error of a GEMM output, per row normwise:
    max over rows of  max_j |C_ij - C_ref_ij| / max_j |C_ref_ij|."""
    got = np.asarray(got, dtype=np.float64)
    den = np.max(np.abs(ref), axis=1, keepdims=True)
    den = np.where(den == 0, 1.0, den)
    return float(np.max(np.abs(got - ref) / den))


def rel_err_elementwise(got, ref):
    """Stricter diagnostic: max |C - C_ref| / max(|C_ref|, rms of the row of
    C_ref).  bf16 output rounding alone reaches 2^-8 = 3.906e-3 here."""
    got = np.asarray(got, dtype=np.float64)
    rms = np.sqrt(np.mean(ref ** 2, axis=1, keepdims=True))
    den = np.maximum(np.abs(ref), rms)
    den = np.where(den == 0, 1.0, den)
    return float(np.max(np.abs(got - ref) / den))


def sample_rows(M, per_band=2, band=128, seed=0):
    """per_band distinct rows from every band of `band` rows (all rows of a
    ragged last band are eligible)."""
    rng = np.random.default_rng(seed)
    out = []
    for b0 in range(0, M, band):
        b1 = min(M, b0 + band)
        out.extend(sorted(rng.choice(np.arange(b0, b1), size=min(per_band, b1 - b0), replace=False)))
    return np.array(out, dtype=np.int64)
