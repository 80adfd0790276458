"""Pins of the oracle GEMM: the exact product of the dequantized FP8 operands
(Eq. 3, paper Sec. 2.2, applied to both operands of the linear layer).
CPU only.

Values of codes come from torch's float8_e4m3fn decoding, not from the
oracle's codec, so the pins are independent of the code they check."""
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle

PAIRS = [(oracle.TENSOR, oracle.TENSOR), (oracle.ROW, oracle.ROW),
         (oracle.BLOCK_1x128, oracle.BLOCK_128x128),
         (oracle.BLOCK_1x128, oracle.BLOCK_1x128)]


def decoded(codes):
    t = torch.from_numpy(np.ascontiguousarray(codes))
    return t.view(torch.float8_e4m3fn).to(torch.float64).numpy()


def random_codes(rng, shape):
    c = rng.integers(0, 256, size=shape, dtype=np.uint8)
    c[(c & 0x7F) == 0x7F] = 0x3A  # no NaN codes
    return c


def random_scales(rng, g, rows, cols):
    n = oracle.scale_count(rows, cols, g)
    # fp32 scales spanning a few decades, arbitrary significands
    return (rng.uniform(0.5, 2.0, n) * 2.0 ** rng.integers(-12, 4, n)).astype(np.float32)


def scale_matrix(s, g, rows, cols):
    """Per-element scale of a [rows, cols] operand (layouts of the oracle)."""
    if g == oracle.TENSOR:
        return np.full((rows, cols), s[0], dtype=np.float64)
    if g == oracle.ROW:
        return np.repeat(s[:, None].astype(np.float64), cols, 1)
    if g == oracle.BLOCK_1x128:
        return np.repeat(s.reshape(cols // 128, rows).T.astype(np.float64), 128, 1)
    if g == oracle.BLOCK_128x128:
        return np.repeat(np.repeat(s.reshape(rows // 128, cols // 128).astype(np.float64),
                                   128, 0), 128, 1)
    raise ValueError(g)


@pytest.mark.parametrize("gA,gB", PAIRS)
@pytest.mark.parametrize("K", [128, 256])
def test_exact_against_fractions(gA, gB, K):
    rng = np.random.default_rng(K + 10 * gA + gB)
    M = 8
    N = 128 if gB == oracle.BLOCK_128x128 else 8
    A, B = random_codes(rng, (M, K)), random_codes(rng, (N, K))
    sA, sB = random_scales(rng, gA, M, K), random_scales(rng, gB, N, K)
    rows = np.arange(M)
    got = oracle.gemm_rows(A, sA, gA, B, sB, gB, rows)
    dA, dB = decoded(A), decoded(B)
    SA, SB = scale_matrix(sA, gA, M, K), scale_matrix(sB, gB, N, K)
    for m in range(M):
        for n in range(0, N, 7 if N > 8 else 1):
            exact = sum(Fraction(SA[m, k]) * Fraction(dA[m, k]) *
                        Fraction(SB[n, k]) * Fraction(dB[n, k]) for k in range(K))
            want = float(exact)  # correctly rounded
            assert got[m, n] == want or abs(Fraction(got[m, n]) - exact) <= \
                abs(exact) * Fraction(1, 2 ** 52), (m, n)


@pytest.mark.parametrize("gA,gB", PAIRS)
def test_matches_fp64_matmul(gA, gB):
    rng = np.random.default_rng(gA * 7 + gB)
    M, N, K = 32, 256, 1024
    A, B = random_codes(rng, (M, K)), random_codes(rng, (N, K))
    sA, sB = random_scales(rng, gA, M, K), random_scales(rng, gB, N, K)
    XA = decoded(A) * scale_matrix(sA, gA, M, K)
    XB = decoded(B) * scale_matrix(sB, gB, N, K)
    ref = XA @ XB.T
    mag = np.abs(XA) @ np.abs(XB).T
    rows = np.array([0, 5, 31, 17])
    got = oracle.gemm_rows(A, sA, gA, B, sB, gB, rows)
    assert np.all(np.abs(got - ref[rows]) <= 1e-13 * mag[rows])


def test_identity_operand_gives_scaled_codes():
    """B = identity codes (1.0 on the diagonal) with power-of-two scales:
    every output is one exact product S_A * S_B * decode(A)."""
    rng = np.random.default_rng(3)
    M, K = 16, 256
    N = K
    A = random_codes(rng, (M, K))
    B = np.zeros((N, K), dtype=np.uint8)
    B[np.arange(N), np.arange(K)] = 0x38
    sA = random_scales(rng, oracle.BLOCK_1x128, M, K)
    sB = (2.0 ** rng.integers(-5, 5, (N // 128) * (K // 128))).astype(np.float32)
    got = oracle.gemm_rows(A, sA, oracle.BLOCK_1x128, B, sB, oracle.BLOCK_128x128,
                           np.arange(M))
    want = decoded(A) * scale_matrix(sA, oracle.BLOCK_1x128, M, K) * \
        scale_matrix(sB, oracle.BLOCK_128x128, N, K).diagonal()[None, :]
    assert np.array_equal(got, want)


def test_rejects_unsupported_pairs():
    A = np.zeros((4, 128), np.uint8)
    s = np.ones(4, np.float32)
    with pytest.raises(ValueError):
        oracle.gemm_rows(A, s, oracle.ROW, A, s, oracle.TENSOR, np.arange(4))
    with pytest.raises(ValueError):
        oracle.gemm_rows(A, s, oracle.BLOCK_128x128, A, s, oracle.BLOCK_128x128,
                         np.arange(4))
