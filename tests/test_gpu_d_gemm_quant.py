"""GPU parity of the GEMM whose epilogue quantizes its own output (Eq. 3
with 1x128 units along N, applied to the bf16 result): the next layer's
activation operand straight out of the GEMM.  Calls go through the C-ABI.

* Where the GEMM's bf16 output is exact (identity weights, power-of-two
  scales), codes and scales must equal the oracle's quantization of the
  oracle's product, bit for bit.
* Elsewhere the bf16 output is fixed by the FP8 matrix instruction's
  arithmetic (tests/csrc/mfma_model.c, pinned by test_gpu_j_mfma_window)
  up to the fp32 roundings on the way, whose bound is known per element:
  where that interval rounds to one bf16 value for all 128 elements of a
  unit, the unit's codes and scale must be exactly the oracle's
  quantization of those bf16 values; in the other units (an element within
  the fp32 bound of a bf16 rounding boundary) the scale must lie between
  those of the smallest and largest possible amax and every code must be
  the oracle's cast of one of its element's possible bf16 values with that
  scale.  The dequantized output is also held to the GEMM tolerance plus
  the E4M3 rounding (2^-4 of the value) per row.
* The fused kernel also gives exactly the bytes of fp8q_gemm followed by
  fp8q_quantize (a consistency check between two entry points)."""
import ctypes
import os

import numpy as np
import pytest
import torch

import oracle
import paper_2609_22870_amd as fp8q
from paper_2609_22870_amd import synth

import _par

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
DEV = "cuda:0"
TOL_DEQ = 2.0 ** -4 + 5e-3


def bf16_round(v):
    """fp64 array -> nearest-even bf16 values (as float64), via fp32."""
    f = np.asarray(v, dtype=np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) >> 16 << 16
    return u.astype(np.uint32).view(np.float32).astype(np.float64)


def to_bf16_bits(v):
    return (np.asarray(v, dtype=np.float32).view(np.uint32) >> 16).astype(np.uint16)


def decode_all(codes):
    table = np.array([oracle.decode(c) for c in range(256)], dtype=np.float64)
    return table[codes]


def scales_matrix_1x128(s, rows, cols):
    return np.repeat(s.reshape(cols // 128, rows).T.astype(np.float64), 128, 1)


def run_fused(A, sA, B, sB):
    codes, scales = fp8q.gemm_quantized(A, sA, fp8q.BLOCK_1x128, B, sB, fp8q.BLOCK_128x128)
    torch.cuda.synchronize()
    return codes, scales


def test_identity_bit_exact():
    M, K = 272, 384
    N = K
    rng = np.random.default_rng(17)
    table = np.array([oracle.decode(c) for c in range(0x7F)], dtype=np.float64)
    vals = table[rng.integers(0, 0x7F, size=(M, K))] * np.where(rng.random((M, K)) < 0.5, -1, 1)
    k = rng.integers(-6, 6, size=(M, K // 128))
    vals[:, ::128] = 448.0
    vals = vals * np.repeat(2.0 ** k, 128, axis=1)
    vals[5, 128:256] = 0.0                    # a zero output unit (S = 1)
    a = torch.from_numpy(vals.astype(np.float32)).to(torch.bfloat16).to(DEV)
    A, sA = fp8q.quantize(a, fp8q.BLOCK_1x128)
    B = torch.zeros((N, K), dtype=torch.uint8, device=DEV)
    B[torch.arange(N), torch.arange(K)] = 0x38
    nb = fp8q.scales_count(N, K, fp8q.BLOCK_128x128)
    sB = torch.from_numpy((2.0 ** rng.integers(-4, 4, size=nb)).astype(np.float32)).to(DEV)
    codes, scales = run_fused(A, sA, B, sB)
    # the oracle's product of its own quantization of the same input
    oA, osA = oracle.quantize(synth.bf16_bits(a.cpu()), oracle.BLOCK_1x128)
    sb = sB.cpu().numpy().reshape(N // 128, K // 128)
    c_ref = decode_all(oA) * scales_matrix_1x128(osA, M, K) * np.repeat(np.diagonal(sb), 128)[None, :]
    assert np.array_equal(bf16_round(c_ref), c_ref)         # exact in bf16
    oc, os_ = oracle.quantize(to_bf16_bits(c_ref), oracle.BLOCK_1x128)
    assert np.array_equal(scales.cpu().numpy().view(np.uint32), os_.view(np.uint32))
    got = codes.cpu().numpy()
    # an exact zero has no sign in the product: compare +0 and -0 codes alike
    got0, oc0 = np.where(got == 0x80, 0, got), np.where(oc == 0x80, 0, oc)
    bad = np.argwhere(got0 != oc0)
    assert bad.size == 0, "codes differ at %s" % bad[:5].tolist()


def fused_vs_oracle(x, w, rows, label):
    print("fused gemm+quantize", label, tuple(x.shape), tuple(w.shape), flush=True)
    A, sA = fp8q.quantize(x, fp8q.BLOCK_1x128)
    B, sB = fp8q.quantize(w, fp8q.BLOCK_128x128)
    codes, scales = run_fused(A, sA, B, sB)
    M, N = A.shape[0], B.shape[0]
    # consistency with the two-call path, every byte
    C = fp8q.gemm(A, sA, fp8q.BLOCK_1x128, B, sB, fp8q.BLOCK_128x128)
    c2, s2 = fp8q.quantize(C, fp8q.BLOCK_1x128)
    torch.cuda.synchronize()
    assert torch.equal(codes, c2)
    assert torch.equal(scales.view(torch.int32), s2.view(torch.int32))
    del C, c2, s2, A, B
    got = codes.cpu().numpy()[rows]
    gs = scales.cpu().numpy().reshape(N // 128, M)[:, rows].T        # [rows][N/128]
    # oracle: quantize the same bf16 inputs, exact product of the sampled rows
    idx = torch.as_tensor(rows, device=x.device)
    oA, osA = _par.quantize(synth.bf16_bits(x[idx].cpu()), oracle.BLOCK_1x128)
    oB, osB = _par.quantize(synth.bf16_bits(w.cpu()), oracle.BLOCK_128x128)
    c_ref = _par.gemm_rows(oA, osA, oracle.BLOCK_1x128, oB, osB, oracle.BLOCK_128x128, np.arange(len(rows)))
    deq = decode_all(got) * np.repeat(gs.astype(np.float64), 128, 1)
    err = _par.rel_err(deq, c_ref)
    print("  dequantized output, max rel err (row normwise) %.3e" % err, flush=True)
    assert err <= TOL_DEQ, err
    check_units(got, gs, oA, osA, oB, osB, K=oA.shape[1])


def bf16_neighbours(lo, hi):
    """The bf16 values RN(x) can take for x in [lo, hi] (RN is monotone):
    RN(lo), the values between, RN(hi); returned as the lower and upper
    ends (float64) and whether they are equal."""
    b_lo, b_hi = bf16_round(lo), bf16_round(hi)
    return b_lo, b_hi, b_lo == b_hi


def check_units(got, gs, oA, osA, oB, osB, K):
    """got: GPU codes [rows, N]; gs: GPU scales [rows, N/128]."""
    rows, N = got.shape
    model, absum, slack = _par.mfma_model(oA, osA, oracle.BLOCK_1x128, oB, osB, oracle.BLOCK_128x128)
    acc = _par.fp32_rounding_factor("promote", K) * absum + slack
    b_lo, b_hi, fixed = bf16_neighbours(model - acc, model + acc)
    unit_fixed = fixed.reshape(rows, N // 128, 128).all(axis=2)
    print("  units whose bf16 output the bound fixes: %d of %d" % (unit_fixed.sum(), unit_fixed.size), flush=True)
    # fixed units: exactly the oracle's quantization of those bf16 values
    oc, osc = oracle.quantize(to_bf16_bits(b_lo), oracle.BLOCK_1x128)
    osc = osc.reshape(N // 128, rows).T
    code_ok = (got == oc).reshape(rows, N // 128, 128).all(axis=2)
    scale_ok = gs.view(np.uint32) == osc.view(np.uint32)
    bad = np.argwhere(unit_fixed & ~(code_ok & scale_ok))
    assert bad.shape[0] == 0, "%d fixed units differ, first (row, unit) %s" % (bad.shape[0], bad[:4].tolist())
    # other units: a possible amax's scale, and each code the cast of one of
    # its element's possible bf16 values with that scale (tests/csrc/unit_check.c)
    check = np.ascontiguousarray(~unit_fixed, dtype=np.uint8)
    first = np.zeros(3, dtype=np.int64)
    ptr = lambda a: a.ctypes.data_as(ctypes.c_void_p)
    lo_bits = np.ascontiguousarray(to_bf16_bits(b_lo))
    hi_bits = np.ascontiguousarray(to_bf16_bits(b_hi))
    got_c = np.ascontiguousarray(got, dtype=np.uint8)
    gs_c = np.ascontiguousarray(gs, dtype=np.float32)
    n_bad = _unit_check()(ptr(lo_bits), ptr(hi_bits), ptr(got_c), ptr(gs_c), ptr(check), rows, N, ptr(first))
    assert n_bad == 0, "%d unfixed units fail, first (row, unit, 1 scale / 2 code) %s" % (n_bad, first.tolist())


_UNIT_CHECK = None


def _unit_check():
    global _UNIT_CHECK
    if _UNIT_CHECK is None:
        from _cbuild import helper
        L = helper("unit_check", link_oracle=True, extra=["-I", os.path.join(ROOT, "oracle")])
        p, i64 = ctypes.c_void_p, ctypes.c_int64
        L.unit_check.argtypes = [p, p, p, p, p, i64, i64, p]
        L.unit_check.restype = i64
        _UNIT_CHECK = L.unit_check
    return _UNIT_CHECK


def test_small_several_tiles_ragged():
    M, K, N = 300, 512, 384
    x = synth.activations(M, K, seed=151, outlier_seed=152, device=DEV)
    w = synth.weights(N, K, seed=153, device=DEV)
    fused_vs_oracle(x, w, np.arange(M), "small ragged")


def test_padded_codes_and_determinism():
    M, K, N = 256, 256, 256
    x = synth.activations(M, K, seed=161, outlier_seed=162, device=DEV)
    w = synth.weights(N, K, seed=163, device=DEV)
    A, sA = fp8q.quantize(x, fp8q.BLOCK_1x128)
    B, sB = fp8q.quantize(w, fp8q.BLOCK_128x128)
    buf = torch.full((M, N + 48), 0x5A, dtype=torch.uint8, device=DEV)
    sc = torch.empty(fp8q.scales_count(M, N, fp8q.BLOCK_1x128), dtype=torch.float32, device=DEV)
    fp8q.gemm_quantized(A, sA, fp8q.BLOCK_1x128, B, sB, fp8q.BLOCK_128x128, codes=buf[:, :N], scales=sc)
    first, first_s = buf.clone(), sc.clone()
    fp8q.gemm_quantized(A, sA, fp8q.BLOCK_1x128, B, sB, fp8q.BLOCK_128x128, codes=buf[:, :N], scales=sc)
    torch.cuda.synchronize()
    assert torch.equal(first, buf) and torch.equal(first_s.view(torch.int32), sc.view(torch.int32))
    assert torch.all(buf[:, N:] == 0x5A)


def test_full_8b_ffn_up():
    """The 8B FFN up-projection forward at full size (256 x 256 tiles),
    sampled rows against the oracle, every byte against the two-call path."""
    M, K, N = 16384, 4096, 12288
    x = synth.activations(M, K, seed=synth.seed_for(2, 0), outlier_seed=synth.seed_for(2, 3), device=DEV)
    w = synth.weights(N, K, seed=synth.seed_for(2, 1), device=DEV)
    fused_vs_oracle(x, w, _par.sample_rows(M), "8B up fwd")
