"""GPU parity of the power-of-two scale variant (not the paper's scale: S
is the smallest power of two with 448 S >= amax) against the oracle, through
the C-ABI: the quantizer bit for bit, and the GEMM whose block scales enter
the matrix instruction as E8M0 exponents to the GEMM tolerance (bit for bit
where the product is exact in bf16)."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_22870_amd as fp8q
from paper_2609_22870_amd import synth

import _par

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
TOL = 4e-3
G_ALL = [fp8q.TENSOR, fp8q.ROW, fp8q.COL, fp8q.BLOCK_1x128, fp8q.BLOCK_128x1, fp8q.BLOCK_128x128]


def check_quantize(x, g, transposed=False, label=""):
    print("pow2 quantize parity", label, tuple(x.shape), "g=%d t=%d" % (g, transposed), flush=True)
    codes, scales = fp8q.quantize(x.to(DEV), g, transposed, pow2=True)
    torch.cuda.synchronize()
    oc, os_ = _par.quantize(synth.bf16_bits(x), g, transposed, pow2=True)
    assert np.array_equal(scales.cpu().numpy().view(np.uint32), os_.view(np.uint32))
    assert np.array_equal(codes.cpu().numpy(), oc)


@pytest.mark.parametrize("g", G_ALL)
@pytest.mark.parametrize("transposed", [False, True])
def test_quantize_all_granularities(g, transposed):
    rows = 256 if g in (fp8q.BLOCK_128x1, fp8q.BLOCK_128x128) else 272
    cols = 384 if g in (fp8q.BLOCK_1x128, fp8q.BLOCK_128x128) else 400
    check_quantize(synth.activations(rows, cols, seed=71 + g, outlier_seed=72 + g), g, transposed, "small")


def test_quantize_extreme_units():
    """Units whose scale clamps at 2^-127 (subnormal amax), units at the
    largest bf16 magnitudes, zero units, and amaxes on both sides of
    448 * 2^k."""
    x = synth.activations(128, 768, seed=73, outlier_seed=74).float()
    x[:, 0:128] *= 2.0 ** -140
    x[:, 128:256] = x[:, 128:256].clamp(-1, 1) * 3.0e38
    x[:, 256:384] = 0.0
    x[:, 384:512] = x[:, 384:512].clamp(-1, 1) * 448.0 * 2.0 ** -20
    x[3, 384] = 448.0 * 2.0 ** -20
    x[4, 640] = 448.0 * 2.0 ** 3 * (1 + 2.0 ** -7)
    check_quantize(x.to(torch.bfloat16), fp8q.BLOCK_1x128, label="extreme units")
    check_quantize(x.to(torch.bfloat16), fp8q.BLOCK_128x128, label="extreme units")


def test_quantize_full_size():
    x = synth.activations(16384, 4096, seed=synth.seed_for(2, 0), outlier_seed=synth.seed_for(2, 3))
    check_quantize(x, fp8q.BLOCK_1x128, label="8B X")
    w = synth.weights(12288, 4096, seed=synth.seed_for(2, 1))
    check_quantize(w, fp8q.BLOCK_128x128, label="8B W")


def gemm_pow2_vs_oracle(x, w, rows=None, label=""):
    print("pow2 gemm parity", label, tuple(x.shape), tuple(w.shape), flush=True)
    A, sA = fp8q.quantize(x, fp8q.BLOCK_1x128, pow2=True)
    B, sB = fp8q.quantize(w, fp8q.BLOCK_128x128, pow2=True)
    C = fp8q.gemm_pow2(A, sA, fp8q.BLOCK_1x128, B, sB, fp8q.BLOCK_128x128)
    torch.cuda.synchronize()
    M = A.shape[0]
    rows = np.arange(M) if rows is None else rows
    got = C.float().cpu().numpy()[rows]
    idx = torch.as_tensor(rows, device=x.device)
    oA, osA = _par.quantize(synth.bf16_bits(x[idx].cpu()), oracle.BLOCK_1x128, pow2=True)
    oB, osB = _par.quantize(synth.bf16_bits(w.cpu()), oracle.BLOCK_128x128, pow2=True)
    ref = _par.gemm_rows(oA, osA, oracle.BLOCK_1x128, oB, osB, oracle.BLOCK_128x128, np.arange(len(rows)))
    # power-of-two scales enter the instruction: the accumulator carries
    # the scaled sum through every K block
    _par.check_gemm(got, ref, oA, osA, oracle.BLOCK_1x128, oB, osB, oracle.BLOCK_128x128, "accumulate",
                    tol=TOL, label=label)


def test_gemm_small_tiles():
    """Shapes that take each tile size, with ragged edges."""
    for (M, K, N) in [(300, 512, 384), (5000, 384, 3072), (8352, 256, 4096)]:   # 64, 128, 256 tiles
        x = synth.activations(M, K, seed=M, outlier_seed=M + 1, device=DEV)
        w = synth.weights(N, K, seed=N, device=DEV)
        rows = np.unique(np.concatenate([np.arange(0, M, max(1, M // 200)), np.arange(M - 8, M)]))
        gemm_pow2_vs_oracle(x, w, rows, "M=%d K=%d N=%d" % (M, K, N))


def test_gemm_identity_bit_exact():
    """B = identity codes with power-of-two scales, A blocks with amax 448 *
    2^k: every output is one exact product, so C = S_A S_B decode(A)."""
    M, K = 160, 384
    N = K
    rng = np.random.default_rng(77)
    table = np.array([oracle.decode(c) for c in range(0x7F)], dtype=np.float64)
    vals = table[rng.integers(0, 0x7F, size=(M, K))] * np.where(rng.random((M, K)) < 0.5, -1, 1)
    k = rng.integers(-6, 6, size=(M, K // 128))
    vals[:, ::128] = 448.0
    vals = vals * np.repeat(2.0 ** k, 128, axis=1)
    a = torch.from_numpy(vals.astype(np.float32)).to(torch.bfloat16).to(DEV)
    A, sA = fp8q.quantize(a, fp8q.BLOCK_1x128, pow2=True)
    B = torch.zeros((N, K), dtype=torch.uint8, device=DEV)
    B[torch.arange(N), torch.arange(K)] = 0x38
    sB = torch.from_numpy((2.0 ** rng.integers(-4, 4, size=(N // 128) * (K // 128))).astype(np.float32)).to(DEV)
    C = fp8q.gemm_pow2(A, sA, fp8q.BLOCK_1x128, B, sB, fp8q.BLOCK_128x128)
    torch.cuda.synchronize()
    oA, osA = oracle.quantize(synth.bf16_bits(a.cpu()), oracle.BLOCK_1x128, pow2=True)
    dA = np.vectorize(oracle.decode)(oA)
    sa_full = np.repeat(osA.reshape(K // 128, M).T.astype(np.float64), 128, 1)
    sb = sB.cpu().numpy().reshape(N // 128, K // 128)
    want = dA * sa_full * np.repeat(np.diagonal(sb), 128)[None, :]
    got = C.float().cpu().numpy()
    assert np.array_equal(got, want)


def test_gemm_full_8b_ffn_up():
    M, K, N = 16384, 4096, 12288
    x = synth.activations(M, K, seed=synth.seed_for(2, 0), outlier_seed=synth.seed_for(2, 3), device=DEV)
    w = synth.weights(N, K, seed=synth.seed_for(2, 1), device=DEV)
    gemm_pow2_vs_oracle(x, w, _par.sample_rows(M), "8B up fwd")


def test_gemm_full_8b_block_gains():
    """Power-of-two block scales that differ by up to 2^12 between the
    weight's 128 x 128 blocks (the synthetic weights alone give one scale
    for nearly every block)."""
    M, K, N = 16384, 4096, 12288
    x = synth.activations(M, K, seed=synth.seed_for(2, 0), outlier_seed=synth.seed_for(2, 3), device=DEV)
    w = synth.weights_block_gains(N, K, seed=synth.seed_for(2, 1), gain_seed=79, device=DEV)
    gemm_pow2_vs_oracle(x, w, rows=_par.sample_rows(M), label="8B up fwd, block gains")
