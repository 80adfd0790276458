"""Two runs of every kernel form give the same bytes (the outputs of a
scaled GEMM are not unique within its tolerance, so run-to-run equality is
asserted on its own): every GEMM launch path (256 x 256 tiles, 128 x 128 tiles of
four and of eight waves, 64 x 64 tiles with and without two K groups) for every scaling
pair, the power-of-two and E5M2 forms, the grouped GEMM and the GEMM with
quantized output; every quantizer granularity plain and transposed
(including the three-kernel tensor, column and transposed row passes), the
dual-layout quantizer and the scale and format variants.  Real synthetic
operands, each run into freshly allocated outputs."""
import pytest
import torch

import paper_2609_22870_amd as fp8q
from paper_2609_22870_amd import synth

pytestmark = pytest.mark.gpu

DEV = "cuda:0"

PAIRS = {
    "tensor": (fp8q.TENSOR, fp8q.TENSOR),
    "row": (fp8q.ROW, fp8q.ROW),
    "block": (fp8q.BLOCK_1x128, fp8q.BLOCK_128x128),
    "blockk": (fp8q.BLOCK_1x128, fp8q.BLOCK_1x128),
}
SHAPES = {
    "256x256 tiles": (8192 + 96, 4096, 4096),
    "128x128 tiles": (4096 + 32, 1024, 1024),
    "128x128 eight-wave tiles": (256 + 32, 2048, 6144),
    "64x64 two K groups": (160, 512, 512),
    "64x64 one K group": (160, 384, 384),
}


def same(a, b):
    return torch.equal(a.contiguous().view(torch.uint8), b.contiguous().view(torch.uint8))


def operands(M, K, N, ga, gb, seed, **kw):
    x = synth.activations(M, K, seed=seed, outlier_seed=seed + 1, device=DEV)
    w = synth.weights(N, K, seed=seed + 2, device=DEV)
    A, sA = fp8q.quantize(x, ga, **kw)
    B, sB = fp8q.quantize(w, gb, **kw)
    return A, sA, B, sB


@pytest.mark.parametrize("shape", list(SHAPES))
@pytest.mark.parametrize("pair", list(PAIRS))
def test_gemm_twice(pair, shape):
    ga, gb = PAIRS[pair]
    M, K, N = SHAPES[shape]
    print("determinism gemm", pair, shape, flush=True)
    A, sA, B, sB = operands(M, K, N, ga, gb, seed=900 + list(SHAPES).index(shape))
    c1 = fp8q.gemm(A, sA, ga, B, sB, gb)
    c2 = fp8q.gemm(A, sA, ga, B, sB, gb)
    torch.cuda.synchronize()
    assert same(c1, c2)


@pytest.mark.parametrize("shape", list(SHAPES))
def test_variant_gemms_twice(shape):
    M, K, N = SHAPES[shape]
    print("determinism pow2 / e5m2 / quantized output", shape, flush=True)
    A, sA, B, sB = operands(M, K, N, fp8q.BLOCK_1x128, fp8q.BLOCK_128x128, seed=920, pow2=True)
    runs = [fp8q.gemm_pow2(A, sA, fp8q.BLOCK_1x128, B, sB, fp8q.BLOCK_128x128) for _ in range(2)]
    torch.cuda.synchronize()
    assert same(*runs)
    A, sA, B, sB = operands(M, K, N, fp8q.BLOCK_1x128, fp8q.BLOCK_128x128, seed=930, e5m2=True)
    for pair in ("block", "blockk"):
        ga, gb = PAIRS[pair]
        if gb == fp8q.BLOCK_1x128:
            B, sB = fp8q.quantize(synth.grads(N, K, seed=931, device=DEV), gb, e5m2=True)
        runs = [fp8q.gemm_formats(A, sA, ga, B, sB, gb, fp8q.A_E5M2 | fp8q.B_E5M2) for _ in range(2)]
        torch.cuda.synchronize()
        assert same(*runs), pair
    if shape in ("256x256 tiles", "128x128 tiles"):
        A, sA, B, sB = operands(M, K, N, fp8q.BLOCK_1x128, fp8q.BLOCK_128x128, seed=940)
        q1 = fp8q.gemm_quantized(A, sA, fp8q.BLOCK_1x128, B, sB, fp8q.BLOCK_128x128)
        q2 = fp8q.gemm_quantized(A, sA, fp8q.BLOCK_1x128, B, sB, fp8q.BLOCK_128x128)
        torch.cuda.synchronize()
        assert same(q1[0], q2[0]) and same(q1[1], q2[1])


@pytest.mark.parametrize("pair", ["tensor", "row", "block"])
def test_grouped_twice(pair):
    ga, gb = PAIRS[pair]
    print("determinism grouped", pair, flush=True)
    M, K = 8192 + 96, 4096
    x = synth.activations(M, K, seed=950, outlier_seed=951, device=DEV)
    A, sA = fp8q.quantize(x, ga)
    probs = []
    for i, n in enumerate((4096, 1024, 1024)):
        B, sB = fp8q.quantize(synth.weights(n, K, seed=952 + i, device=DEV), gb)
        probs.append((A, sA, B, sB))
    r1 = fp8q.gemm_grouped(probs, ga, gb)
    r2 = fp8q.gemm_grouped(probs, ga, gb)
    torch.cuda.synchronize()
    for a, b in zip(r1, r2):
        assert same(a, b)


G_ALL = [fp8q.TENSOR, fp8q.ROW, fp8q.COL, fp8q.BLOCK_1x128, fp8q.BLOCK_128x1, fp8q.BLOCK_128x128]


@pytest.mark.parametrize("flags", [{}, {"pow2": True}, {"e5m2": True}])
@pytest.mark.parametrize("transposed", [False, True])
@pytest.mark.parametrize("g", G_ALL)
def test_quantizer_twice(g, transposed, flags):
    """4096 x 6144: many workgroups per unit for the tensor, column and
    transposed row passes (partial maxima, their reduction, the cast)."""
    x = synth.activations(4096, 6144, seed=960 + g, outlier_seed=961, device=DEV)
    r1 = fp8q.quantize(x, g, transposed, **flags)
    r2 = fp8q.quantize(x, g, transposed, **flags)
    torch.cuda.synchronize()
    assert same(r1[0], r2[0]) and same(r1[1], r2[1])


@pytest.mark.parametrize("flags", [{}, {"pow2": True}, {"e5m2": True}])
def test_dual_twice(flags):
    x = synth.grads(4096, 6144, seed=970, device=DEV)
    r1 = fp8q.quantize_dual(x, **flags)
    r2 = fp8q.quantize_dual(x, **flags)
    torch.cuda.synchronize()
    for a, b in zip(r1, r2):
        assert same(a, b)
