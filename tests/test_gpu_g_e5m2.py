"""GPU parity of the E5M2 variant for gradients (the paper leaves the FP8
format of Eq. 3 open; F_max = 57344) against the oracle, through the C-ABI:
the device cast over every fp32 pattern, the quantizer (single and dual
layout) bit for bit, and the GEMM with E5M2 operands in the backward layouts
to the GEMM tolerance (bit for bit where the product is exact in bf16)."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_22870_amd as fp8q
from paper_2609_22870_amd import synth

import _par
from test_gpu_a_quantize import all_bf16_pairs

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
TOL = 4e-3
G_ALL = [fp8q.TENSOR, fp8q.ROW, fp8q.COL, fp8q.BLOCK_1x128, fp8q.BLOCK_128x1, fp8q.BLOCK_128x128]


def check_quantize(x, g, transposed=False, pow2=False, label=""):
    print("e5m2 quantize parity", label, tuple(x.shape), "g=%d t=%d pow2=%d" % (g, transposed, pow2), flush=True)
    codes, scales = fp8q.quantize(x.to(DEV), g, transposed, pow2=pow2, e5m2=True)
    torch.cuda.synchronize()
    oc, os_ = _par.quantize(synth.bf16_bits(x.cpu()), g, transposed, pow2=pow2, e5m2=True)
    assert np.array_equal(scales.cpu().numpy().view(np.uint32), os_.view(np.uint32))
    assert np.array_equal(codes.cpu().numpy(), oc)


def test_cast_f32_all_patterns():
    """The device E5M2 rounding routine on all 2^32 fp32 patterns (scale 1),
    NaN inputs excluded, in 2^28-pattern chunks."""
    chunk = 1 << 28
    for start in range(0, 1 << 32, chunk):
        print("e5m2 cast sweep chunk", hex(start), flush=True)
        bits = np.arange(start, start + chunk, dtype=np.uint64).astype(np.uint32)
        x = torch.from_numpy(bits.view(np.int32)).view(torch.float32)
        got = fp8q.cast_f32(x.to(DEV), 1.0, e5m2=True).cpu().numpy()
        vals = bits.view(np.float32)
        keep = ~np.isnan(vals)
        want = _par.cast_f32(vals, 1.0, e5m2=True)
        assert np.array_equal(got[keep], want[keep]), hex(start)


@pytest.mark.parametrize("scale", [0.37, 3.0e-9, 1.7e30])
def test_cast_f32_scaled(scale):
    rng = np.random.default_rng(9)
    x = (rng.standard_normal(1 << 20) * 57344 * scale).astype(np.float32)
    got = fp8q.cast_f32(torch.from_numpy(x).to(DEV), scale, e5m2=True).cpu().numpy()
    assert np.array_equal(got, oracle.cast_f32(x, scale, e5m2=True))


@pytest.mark.parametrize("g", G_ALL)
@pytest.mark.parametrize("transposed", [False, True])
def test_quantize_all_granularities(g, transposed):
    rows = 256 if g in (fp8q.BLOCK_128x1, fp8q.BLOCK_128x128) else 272
    cols = 384 if g in (fp8q.BLOCK_1x128, fp8q.BLOCK_128x128) else 400
    check_quantize(synth.grads(rows, cols, seed=81 + g), g, transposed, label="small")


@pytest.mark.parametrize("g", [fp8q.BLOCK_1x128, fp8q.BLOCK_128x1, fp8q.BLOCK_128x128, fp8q.ROW])
def test_quantize_pow2_scales(g):
    check_quantize(synth.grads(256, 384, seed=91 + g), g, pow2=True, label="pow2")


def test_exhaustive_bf16_amax_x_pairs():
    """Every (bf16 amax, bf16 x) pair of the 1x128 path, E5M2 codes."""
    x = all_bf16_pairs(DEV)
    print("e5m2 exhaustive pairs: rows", x.shape[0], flush=True)
    codes, scales = fp8q.quantize(x, fp8q.BLOCK_1x128, e5m2=True)
    torch.cuda.synchronize()
    gc, gs = codes.cpu().numpy(), scales.cpu().numpy()
    bits = synth.bf16_bits(x)
    del codes, scales, x
    oc, os_ = _par.quantize(bits, oracle.BLOCK_1x128, e5m2=True)
    assert np.array_equal(gs.view(np.uint32), os_.view(np.uint32))
    assert np.array_equal(gc, oc)


@pytest.mark.parametrize("pow2", [False, True])
def test_dual_layout(pow2):
    """The dual quantizer with E5M2 codes equals the two single-layout calls
    byte for byte, and the oracle."""
    dy = synth.grads(384, 640, seed=95, device=DEV)
    print("e5m2 dual parity pow2=%d" % pow2, flush=True)
    cr, sr, ct, st = fp8q.quantize_dual(dy, pow2=pow2, e5m2=True)
    c1, s1 = fp8q.quantize(dy, fp8q.BLOCK_1x128, pow2=pow2, e5m2=True)
    c2, s2 = fp8q.quantize(dy, fp8q.BLOCK_128x1, True, pow2=pow2, e5m2=True)
    torch.cuda.synchronize()
    assert torch.equal(cr, c1) and torch.equal(sr, s1) and torch.equal(ct, c2) and torch.equal(st, s2)
    oc, os_ = _par.quantize(synth.bf16_bits(dy.cpu()), oracle.BLOCK_1x128, pow2=pow2, e5m2=True)
    assert np.array_equal(cr.cpu().numpy(), oc) and np.array_equal(sr.cpu().numpy(), os_)
    oc, os_ = _par.quantize(synth.bf16_bits(dy.cpu()), oracle.BLOCK_128x1, True, pow2=pow2, e5m2=True)
    assert np.array_equal(ct.cpu().numpy(), oc) and np.array_equal(st.cpu().numpy(), os_)


def test_quantize_full_32b_dy():
    """The 32B FFN up-projection's output gradient, 16384 x 25600: 1x128 for
    dgrad and 128x1 transposed for wgrad, both from the dual quantizer."""
    dy = synth.grads(16384, 25600, seed=synth.seed_for(5, 2), device=DEV)
    print("e5m2 dual 32B dY", flush=True)
    cr, sr, ct, st = fp8q.quantize_dual(dy, e5m2=True)
    torch.cuda.synchronize()
    bits = synth.bf16_bits(dy.cpu())
    del dy
    oc, os_ = _par.quantize(bits, oracle.BLOCK_1x128, e5m2=True)
    assert np.array_equal(sr.cpu().numpy(), os_) and np.array_equal(cr.cpu().numpy(), oc)
    del oc, os_, cr, sr
    oc, os_ = _par.quantize(bits, oracle.BLOCK_128x1, True, e5m2=True)
    assert np.array_equal(st.cpu().numpy(), os_) and np.array_equal(ct.cpu().numpy(), oc)


# ---- GEMM with E5M2 operands

def run_formats(a_src, b_src, ga, gb, fa, fb, a_t=False, b_t=False, rows=None, label=""):
    """Quantize a_src (E5M2 if fa) and b_src (E5M2 if fb), optionally
    transposed as the backward layouts need, multiply through
    fp8q_gemm_formats and compare the listed rows with the oracle."""
    print("e5m2 gemm parity", label, tuple(a_src.shape), tuple(b_src.shape), "fa=%d fb=%d" % (fa, fb), flush=True)
    qa = fp8q.BLOCK_128x1 if a_t else ga
    qb = (fp8q.BLOCK_128x1 if gb == fp8q.BLOCK_1x128 else gb) if b_t else gb
    A, sA = fp8q.quantize(a_src, qa, a_t, e5m2=bool(fa))
    B, sB = fp8q.quantize(b_src, qb, b_t, e5m2=bool(fb))
    C = fp8q.gemm_formats(A, sA, ga, B, sB, gb, (fp8q.A_E5M2 if fa else 0) | (fp8q.B_E5M2 if fb else 0))
    torch.cuda.synchronize()
    M = A.shape[0]
    rows = np.arange(M) if rows is None else rows
    got = C.float().cpu().numpy()[rows]
    del C, A, B, sA, sB
    idx = torch.as_tensor(rows, device=a_src.device)
    a_cpu = (a_src[:, idx] if a_t else a_src[idx]).contiguous().cpu()
    oA, osA = _par.quantize(synth.bf16_bits(a_cpu), qa, a_t, e5m2=bool(fa))
    oB, osB = _par.quantize(synth.bf16_bits(b_src.cpu()), qb, b_t, e5m2=bool(fb))
    ref = _par.gemm_rows(oA, osA, ga, oB, osB, gb, np.arange(len(rows)),
                         fmtA=oracle.FMT_E5M2 if fa else oracle.FMT_E4M3,
                         fmtB=oracle.FMT_E5M2 if fb else oracle.FMT_E4M3)
    return _par.check_gemm(got, ref, oA, osA, ga, oB, osB, gb, "promote",
                           fmtA=oracle.FMT_E5M2 if fa else oracle.FMT_E4M3,
                           fmtB=oracle.FMT_E5M2 if fb else oracle.FMT_E4M3, tol=TOL, label=label)


# (tokens, layer input width = dX columns, layer output width = contraction)
@pytest.mark.parametrize("T,K_l,N_l", [(300, 384, 512), (5000, 3072, 384), (8352, 4096, 256)])  # 64, 128, 256 tiles
def test_dgrad_e5m2_dy_all_tiles(T, K_l, N_l):
    """dX[T, K_l] = dY[T, N_l] W[N_l, K_l]: A = dY in E5M2 (1x128), B = W^T
    (128x128, E4M3, written transposed)."""
    dy = synth.grads(T, N_l, seed=T + 1, device=DEV)
    w = synth.weights(N_l, K_l, seed=N_l + 2, device=DEV)
    rows = np.unique(np.concatenate([np.arange(0, T, max(1, T // 160)), np.arange(T - 8, T)]))
    run_formats(dy, w, fp8q.BLOCK_1x128, fp8q.BLOCK_128x128, 1, 0, b_t=True, rows=rows,
                label="dgrad T=%d" % T)


@pytest.mark.parametrize("T,K_l,N_l", [(512, 256, 384), (1024, 2048, 2560)])   # 64 and 128 tiles
def test_wgrad_e5m2_dy(T, K_l, N_l):
    """dW^T[K_l, N_l] = X^T dY: A = X^T (E4M3), B = dY^T (E5M2), both grouped
    by 128 along the tokens and written transposed."""
    x = synth.activations(T, K_l, seed=T + 3, outlier_seed=T + 4, device=DEV)
    dy = synth.grads(T, N_l, seed=T + 5, device=DEV)
    run_formats(x, dy, fp8q.BLOCK_1x128, fp8q.BLOCK_1x128, 0, 1, a_t=True, b_t=True, label="wgrad T=%d" % T)


def test_wgrad_dy_as_a():
    """dW[N_l, K_l] = dY^T X with the gradient as A (formats A_E5M2)."""
    T, K_l, N_l = 768, 384, 256
    x = synth.activations(T, K_l, seed=131, outlier_seed=132, device=DEV)
    dy = synth.grads(T, N_l, seed=133, device=DEV)
    run_formats(dy, x, fp8q.BLOCK_1x128, fp8q.BLOCK_1x128, 1, 0, a_t=True, b_t=True, label="wgrad dY as A")


def test_both_operands_e5m2():
    a = synth.grads(640, 512, seed=141, device=DEV)
    b = synth.grads(384, 512, seed=142, device=DEV)
    run_formats(a, b, fp8q.BLOCK_1x128, fp8q.BLOCK_128x128, 1, 1, label="E5M2 x E5M2")
    run_formats(a, b, fp8q.BLOCK_1x128, fp8q.BLOCK_1x128, 1, 1, label="E5M2 x E5M2, 1x128 pair")


def test_identity_bit_exact_e5m2():
    """A in E5M2 with power-of-two block scales (amax 57344 * 2^k), B = E4M3
    identity codes with power-of-two scales: every output is one exact
    product, so C = S_A S_B decode(A) bit for bit."""
    M, K = 160, 384
    rng = np.random.default_rng(151)
    table = np.array([oracle.decode_e5m2(c) for c in range(0x7C)], dtype=np.float64)
    vals = table[rng.integers(0, 0x7C, size=(M, K))] * np.where(rng.random((M, K)) < 0.5, -1, 1)
    k = rng.integers(-20, 4, size=(M, K // 128))
    vals[:, ::128] = 57344.0
    vals = vals * np.repeat(2.0 ** k, 128, axis=1)
    a = torch.from_numpy(vals.astype(np.float32)).to(torch.bfloat16).to(DEV)
    assert torch.equal(a.float().cpu(), torch.from_numpy(vals.astype(np.float32)))
    A, sA = fp8q.quantize(a, fp8q.BLOCK_1x128, e5m2=True)
    B = torch.zeros((K, K), dtype=torch.uint8, device=DEV)
    B[torch.arange(K), torch.arange(K)] = 0x38
    sB = torch.from_numpy((2.0 ** rng.integers(-4, 4, size=(K // 128) ** 2)).astype(np.float32)).to(DEV)
    C = fp8q.gemm_formats(A, sA, fp8q.BLOCK_1x128, B, sB, fp8q.BLOCK_128x128, fp8q.A_E5M2)
    torch.cuda.synchronize()
    oA, osA = oracle.quantize(synth.bf16_bits(a.cpu()), oracle.BLOCK_1x128, e5m2=True)
    sa = osA.reshape(K // 128, M).T.astype(np.float64)
    assert np.array_equal(sa, 2.0 ** k)
    dA = np.vectorize(oracle.decode_e5m2)(oA)
    sb = sB.cpu().numpy().reshape(K // 128, K // 128)
    want = dA * np.repeat(sa, 128, 1) * np.repeat(np.diagonal(sb), 128)[None, :]
    assert np.array_equal(C.float().cpu().numpy(), want)


@pytest.mark.parametrize("pas", ["dgrad", "wgrad"])
def test_full_32b_up_backward(pas):
    """The 32B FFN up-projection's backward GEMMs with dY in E5M2: dgrad
    16384 x 25600 -> 5120 and wgrad over 16384 tokens (sampled rows)."""
    T, k_in, n_out = 16384, 5120, 25600
    w = synth.weights(n_out, k_in, seed=synth.seed_for(5, 1), device=DEV)
    dy = synth.grads(T, n_out, seed=synth.seed_for(5, 2), device=DEV)
    if pas == "dgrad":
        run_formats(dy, w, fp8q.BLOCK_1x128, fp8q.BLOCK_128x128, 1, 0, b_t=True,
                    rows=_par.sample_rows(T), label="32B up dgrad")
    else:
        x = synth.activations(T, k_in, seed=synth.seed_for(5, 0), outlier_seed=synth.seed_for(5, 3), device=DEV)
        del w
        run_formats(x, dy, fp8q.BLOCK_1x128, fp8q.BLOCK_1x128, 0, 1, a_t=True, b_t=True,
                    rows=_par.sample_rows(k_in), label="32B up wgrad")
