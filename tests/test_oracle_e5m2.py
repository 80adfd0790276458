"""Pins of the oracle's E5M2 variant (gradient codes; the paper leaves the
FP8 format of Eq. 3, Sec. 2.2, open): the codec against the OCP E5M2
definition, an independent encoder, brute force and torch's float8_e5m2;
the quantizer with F_max = 57344 against torch routines and the
invariants of Eq. 3; the GEMM with E5M2 operands against exact rational
arithmetic.  CPU only."""
import ctypes
import math
import os
import struct
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle
from paper_2609_22870_amd import synth

from _cbuild import helper

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "e5m2_key_values.txt")
FMAX = 57344.0
G_ALL = [oracle.TENSOR, oracle.ROW, oracle.COL, oracle.BLOCK_1x128,
         oracle.BLOCK_128x1, oracle.BLOCK_128x128]


def f32(b):
    return struct.unpack("<f", struct.pack("<I", b))[0]


def torch_decode_all():
    codes = torch.arange(256, dtype=torch.int32).to(torch.uint8)
    return codes.view(torch.float8_e5m2).to(torch.float64).numpy()


# ---- codec

def test_golden_key_values():
    with open(GOLDEN) as fh:
        rows = [ln.split("#")[0].split() for ln in fh if ln.strip() and not ln.startswith("#")]
    assert len(rows) == 13
    for code_hex, val in rows:
        got = oracle.decode_e5m2(int(code_hex, 16))
        if val == "nan":
            assert math.isnan(got)
        else:
            want = float(val)
            assert got == want and math.copysign(1, got) == math.copysign(1, want), code_hex


def test_decode_all_256_matches_torch():
    ref = torch_decode_all()
    for c in range(256):
        got = oracle.decode_e5m2(c)
        if math.isnan(ref[c]):
            assert math.isnan(got), c
        else:
            assert got == ref[c] and math.copysign(1, got) == math.copysign(1, ref[c]), c
    assert sum(math.isnan(oracle.decode_e5m2(c)) for c in range(256)) == 6
    assert sum(math.isinf(oracle.decode_e5m2(c)) for c in range(256)) == 2


def test_decode_monotone_and_distinct():
    vals = [oracle.decode_e5m2(c) for c in range(0x7C)]
    assert all(a < b for a, b in zip(vals, vals[1:]))
    assert vals[-1] == FMAX and vals[1] == 2.0 ** -16 and vals[4] == 2.0 ** -14
    for c in range(0x7C):
        assert oracle.decode_e5m2(c | 0x80) == -vals[c]


def test_encode_decode_roundtrip_finite_codes():
    for c in list(range(0x7C)) + list(range(0x80, 0xFC)):
        assert oracle.encode_e5m2(oracle.decode_e5m2(c)) == c, hex(c)
    assert oracle.encode_e5m2(-0.0) == 0x80 and oracle.encode_e5m2(0.0) == 0x00


def test_midpoints_ties_to_even_and_neighbours():
    vals = [oracle.decode_e5m2(c) for c in range(0x7C)]
    for c in range(0x7B):
        lo, hi = vals[c], vals[c + 1]
        mid = np.float32((lo + hi) / 2)
        assert float(mid) == (lo + hi) / 2
        even = c if c % 2 == 0 else c + 1
        assert oracle.encode_e5m2(float(mid)) == even, hex(c)
        assert oracle.encode_e5m2(-float(mid)) == even | 0x80
        up = np.nextafter(mid, np.float32(np.inf), dtype=np.float32)
        dn = np.nextafter(mid, np.float32(0), dtype=np.float32)
        assert oracle.encode_e5m2(float(up)) == c + 1
        assert oracle.encode_e5m2(float(dn)) == c


def test_saturation_never_gives_infinity():
    for v in [FMAX, 57345.0, 61439.99, 61440.0, 61441.0, 65536.0, 1e6, 3.0e38,
              f32(0x7F7FFFFF), math.inf]:
        assert oracle.encode_e5m2(v) == 0x7B, v
        assert oracle.encode_e5m2(-v) == 0xFB, v


def test_exhaustive_against_independent_encoder():
    """Every fp32 pattern with magnitude in [2^-19, 2^17), plus every 97th
    elsewhere; FP8_FULL_SWEEP=1 walks all 2^32 patterns."""
    lib = helper("e5m2_sweep", link_oracle=True)
    lib.sweep.argtypes = [ctypes.c_uint64, ctypes.c_uint64, ctypes.c_uint64,
                          ctypes.c_int, ctypes.POINTER(ctypes.c_uint64),
                          ctypes.POINTER(ctypes.c_uint32)]
    lib.sweep.restype = ctypes.c_uint64
    threads = min(16, len(os.sched_getaffinity(0)))
    checked, first = ctypes.c_uint64(), ctypes.c_uint32()

    def run(start, end, stride):
        bad = lib.sweep(start, end, stride, threads, ctypes.byref(checked), ctypes.byref(first))
        assert bad == 0, "mismatch at 0x%08x" % first.value
        return checked.value

    if os.environ.get("FP8_FULL_SWEEP") == "1":
        assert run(0, 1 << 32, 1) == (1 << 32) - 2 * ((1 << 23) - 1)
        return
    lo, hi = (127 - 19) << 23, (127 + 17) << 23
    n = 0
    for sign in (0, 1 << 31):
        n += run(sign | lo, sign | hi, 1)
        n += run(sign, sign | lo, 97)
        n += run(sign | hi, sign | 0x7FFFFFFF, 97)
    assert n > 2 * (hi - lo)


def test_brute_force_sample():
    table = [oracle.decode_e5m2(c) for c in range(0x7C)]
    rng = np.random.default_rng(17)
    vals = [f32(int(b)) for b in rng.integers(0, 1 << 32, size=3000, dtype=np.uint64)]
    vals += list(rng.uniform(-7e4, 7e4, 2000)) + list(rng.uniform(-1e-4, 1e-4, 2000))
    for v in vals:
        v = float(np.float32(v))
        if math.isnan(v):
            continue
        a, sign = abs(v), (0x80 if math.copysign(1, v) < 0 else 0)
        if a >= FMAX:
            want = sign | 0x7B
        else:
            best, bestd = None, None
            for c, t in enumerate(table):
                d = abs(a - t)
                if bestd is None or d < bestd or (d == bestd and c % 2 == 0):
                    best, bestd = c, d
            want = sign | best
        assert oracle.encode_e5m2(v) == want, v


def test_matches_torch_cast_in_range():
    """torch's float8_e5m2 conversion rounds to nearest even; compared where
    no saturation is needed (|v| <= 57344)."""
    rng = np.random.default_rng(19)
    x = np.concatenate([rng.standard_normal(200000).astype(np.float32) * 1e4,
                        rng.standard_normal(200000).astype(np.float32) * 1e-5,
                        rng.uniform(-FMAX, FMAX, 200000).astype(np.float32)])
    x = x[np.abs(x) <= FMAX]
    want = torch.from_numpy(x).to(torch.float8_e5m2).view(torch.uint8).numpy()
    assert np.array_equal(oracle.cast_f32(x, 1.0, e5m2=True), want)


# ---- quantizer with F_max = 57344

def units_of(xf, g):
    R, C = xf.shape
    if g == oracle.TENSOR:
        return xf.reshape(1, 1, R * C)
    if g == oracle.ROW:
        return xf.reshape(R, 1, C)
    if g == oracle.COL:
        return xf.t().reshape(C, 1, R)
    if g == oracle.BLOCK_1x128:
        return xf.reshape(R, C // 128, 128).permute(1, 0, 2)
    if g == oracle.BLOCK_128x1:
        return xf.reshape(R // 128, 128, C).permute(0, 2, 1)
    u = xf.reshape(R // 128, 128, C // 128, 128).permute(0, 2, 1, 3)
    return u.reshape(R // 128, C // 128, 128 * 128)


def codes_back(q, g, R, C):
    if g in (oracle.TENSOR, oracle.ROW):
        return q.reshape(R, C)
    if g == oracle.COL:
        return q.reshape(C, R).t()
    if g == oracle.BLOCK_1x128:
        return q.permute(1, 0, 2).reshape(R, C)
    if g == oracle.BLOCK_128x1:
        return q.permute(0, 2, 1).reshape(R, C)
    return q.reshape(R // 128, C // 128, 128, 128).permute(0, 2, 1, 3).reshape(R, C)


def torch_reference(x, g):
    """Scales and E5M2 codes by torch routines (amax by reshaping into
    units, fp32 division, torch's float8_e5m2 cast)."""
    xf = x.float()
    units = units_of(xf, g)
    s = units.abs().amax(dim=-1, keepdim=True) / FMAX
    s = torch.where(s == 0, torch.ones_like(s), s)
    q = (units / s).to(torch.float8_e5m2).view(torch.uint8)
    return codes_back(q, g, *xf.shape).contiguous().numpy(), s.reshape(-1).numpy()


def grads(rows, cols, seed):
    """Output-gradient-like values: N(0, 1e-3) with 1% of columns x50."""
    return synth.normal_bf16((rows, cols), 1e-3, seed, outlier_cols=synth.outlier_columns(cols, seed + 1))


@pytest.mark.parametrize("g", G_ALL)
def test_quantize_matches_torch_reference(g):
    x = grads(256, 384, 31)
    codes, scales = oracle.quantize(synth.bf16_bits(x), g, e5m2=True)
    rc, rs = torch_reference(x, g)
    assert np.array_equal(scales, rs)
    assert np.array_equal(codes, rc)


@pytest.mark.parametrize("g", G_ALL)
def test_transposed_output_is_the_byte_transpose(g):
    x = grads(256, 384, 33)
    codes, scales = oracle.quantize(synth.bf16_bits(x), g, transposed=True, e5m2=True)
    c0, s0 = oracle.quantize(synth.bf16_bits(x), g, e5m2=True)
    assert np.array_equal(codes, c0.T)
    assert np.array_equal(np.sort(scales), np.sort(s0))


def test_amax_element_encodes_to_57344():
    """For every positive finite bf16 amax a but one, the element equal to a
    encodes to 0x7B.  The exception is a = 2^-131: S = RN32(2^-131 / 57344)
    is the fp32 subnormal 5 * 2^-149, so a / S = 2^18 / 5 = 52428.8, which
    is below the midpoint 53248 of 49152 and 57344 and encodes to 0x7A (the
    definition, with S that deep in the subnormals, loses the top code)."""
    a = np.arange(1, 0x7F80, dtype=np.uint16)
    x = np.zeros((a.size, 128), dtype=np.uint16)
    x[:, 5] = a
    x[:, 6] = a | 0x8000
    codes, scales = oracle.quantize(x, oracle.ROW, e5m2=True)
    odd = a == 0x0004                                  # bf16 bits of 2^-131
    assert f32(0x0004 << 16) == 2.0 ** -131
    assert np.all(codes[~odd, 5] == 0x7B) and np.all(codes[~odd, 6] == 0xFB)
    assert scales[odd][0] == np.float32(5 * 2.0 ** -149)
    assert codes[odd, 5][0] == 0x7A and codes[odd, 6][0] == 0xFA


def test_ties_through_the_whole_path():
    """amax = 57344 * 2^k gives S = 2^k exactly: midpoints between E5M2
    neighbours scaled by 2^k go to the even code."""
    table = [oracle.decode_e5m2(c) for c in range(0x7C)]
    mids = [(table[c] + table[c + 1]) / 2 for c in range(0x7B)]
    want = [c if c % 2 == 0 else c + 1 for c in range(0x7B)]
    for k in (-30, 0, 20):
        vals = [m * 2.0 ** k for m in mids] + [FMAX * 2.0 ** k]
        vals += [-v for v in vals[: 128 - len(vals)]]
        t = torch.tensor(vals[:128], dtype=torch.float32)
        assert torch.equal(t.to(torch.bfloat16).float(), t)
        codes, scales = oracle.quantize(synth.bf16_bits(t.to(torch.bfloat16).reshape(1, -1)),
                                        oracle.BLOCK_1x128, e5m2=True)
        assert scales[0] == 2.0 ** k
        assert list(codes[0, :0x7B]) == want and codes[0, 0x7B] == 0x7B
        assert list(codes[0, 0x7C:]) == [w | 0x80 for w in want[: 128 - 0x7C]]


@pytest.mark.parametrize("g", G_ALL)
def test_dequantization_error_bound(g):
    """Half an E5M2 step: 2^-3 relative for normals, 2^-17 absolute (times
    S) in the subnormal range, plus the fp32 rounding of the quotient."""
    x = grads(256, 256, 35)
    codes, scales = oracle.quantize(synth.bf16_bits(x), g, e5m2=True)
    table = np.array([oracle.decode_e5m2(c) for c in range(256)])
    dec = table[codes]
    assert np.all(np.isfinite(dec)) and np.all(np.abs(dec) <= FMAX)
    xf = x.float().numpy().astype(np.float64)
    u = units_of(x.float(), g)
    su = u.abs().amax(dim=-1, keepdim=True) / FMAX
    su = torch.where(su == 0, torch.ones_like(su), su)
    s_full = codes_back(su.expand_as(u).contiguous(), g, *x.shape).double().numpy()
    assert np.array_equal(np.unique(s_full), np.unique(scales.astype(np.float64)))
    q = xf / s_full
    bound = s_full * (np.maximum(2.0 ** -3 * np.abs(dec), 2.0 ** -17) + 2.0 ** -23 * np.abs(q))
    assert np.all(np.abs(xf - s_full * dec) <= bound)


@pytest.mark.parametrize("j", [-40, 7])
def test_power_of_two_scale_invariance(j):
    x = grads(256, 256, 37)
    y = (x.float() * 2.0 ** j).to(torch.bfloat16)
    assert torch.equal(y.float(), x.float() * 2.0 ** j)
    cx, sx = oracle.quantize(synth.bf16_bits(x), oracle.BLOCK_1x128, e5m2=True)
    cy, sy = oracle.quantize(synth.bf16_bits(y), oracle.BLOCK_1x128, e5m2=True)
    assert np.array_equal(cx, cy)
    assert np.array_equal(sy, (sx.astype(np.float64) * 2.0 ** j).astype(np.float32))


def test_pow2_scale_with_e5m2_against_exact_search():
    """The two variants together: S is the smallest power of two with
    57344 S >= amax (at least 2^-127)."""
    for amax in [FMAX * 2.0 ** k for k in range(-20, 20)] + [1.0, 3.0, 1.75 * 2.0 ** -100,
                                                             2.0 ** -133, 3.3895313892515355e38]:
        x = torch.tensor([[amax, -amax / 8]], dtype=torch.float32).to(torch.bfloat16)
        a = Fraction(float(x.float().abs().max()))
        k = -200
        while FMAX * Fraction(2) ** k < a:
            k += 1
        _, s = oracle.quantize(synth.bf16_bits(x), oracle.TENSOR, pow2=True, e5m2=True)
        assert float(s[0]) == float(Fraction(2) ** max(k, -127)), amax


# ---- GEMM with E5M2 operands

def decoded(codes, e5m2):
    t = torch.from_numpy(np.ascontiguousarray(codes))
    return t.view(torch.float8_e5m2 if e5m2 else torch.float8_e4m3fn).to(torch.float64).numpy()


def random_codes(rng, shape, e5m2):
    c = rng.integers(0, 256, size=shape, dtype=np.uint8)
    if e5m2:
        c[(c & 0x7F) >= 0x7C] = 0x3D    # no infinities or NaNs
    else:
        c[(c & 0x7F) == 0x7F] = 0x3A
    return c


@pytest.mark.parametrize("fa,fb", [(1, 0), (0, 1), (1, 1)])
@pytest.mark.parametrize("gA,gB", [(oracle.BLOCK_1x128, oracle.BLOCK_128x128),
                                   (oracle.BLOCK_1x128, oracle.BLOCK_1x128),
                                   (oracle.TENSOR, oracle.TENSOR)])
def test_gemm_exact_against_fractions(fa, fb, gA, gB):
    rng = np.random.default_rng(100 * fa + 10 * fb + gA + gB)
    M, K = 4, 256
    N = 128 if gB == oracle.BLOCK_128x128 else 6
    A, B = random_codes(rng, (M, K), fa), random_codes(rng, (N, K), fb)

    def scales(g, rows, cols):
        n = oracle.scale_count(rows, cols, g)
        return (rng.uniform(0.5, 2.0, n) * 2.0 ** rng.integers(-20, 4, n)).astype(np.float32)

    sA, sB = scales(gA, M, K), scales(gB, N, K)
    got = oracle.gemm_rows(A, sA, gA, B, sB, gB, np.arange(M), fmtA=fa, fmtB=fb)
    dA, dB = decoded(A, fa), decoded(B, fb)

    def sc(s, g, r, k, rows, cols):
        if g == oracle.TENSOR:
            return s[0]
        if g == oracle.BLOCK_1x128:
            return s[(k // 128) * rows + r]
        return s[(r // 128) * (cols // 128) + k // 128]

    for m in range(M):
        for n in range(0, N, 11 if N > 8 else 1):
            exact = sum(Fraction(float(sc(sA, gA, m, k, M, K))) * Fraction(dA[m, k]) *
                        Fraction(float(sc(sB, gB, n, k, N, K))) * Fraction(dB[n, k]) for k in range(K))
            assert abs(Fraction(got[m, n]) - exact) <= abs(exact) * Fraction(1, 2 ** 52), (m, n)


def test_gemm_identity_operand_with_e5m2_codes():
    """B = identity (E4M3 1.0) with power-of-two scales and A in E5M2: each
    output is one exact product S_A S_B decode(A)."""
    rng = np.random.default_rng(41)
    M, K = 8, 256
    A = random_codes(rng, (M, K), True)
    B = np.zeros((K, K), dtype=np.uint8)
    B[np.arange(K), np.arange(K)] = 0x38
    sA = (rng.uniform(0.5, 2.0, M * 2) * 2.0 ** rng.integers(-10, 4, M * 2)).astype(np.float32)
    sB = (2.0 ** rng.integers(-5, 5, 4)).astype(np.float32)
    got = oracle.gemm_rows(A, sA, oracle.BLOCK_1x128, B, sB, oracle.BLOCK_128x128, np.arange(M),
                           fmtA=oracle.FMT_E5M2)
    sa_full = np.repeat(sA.reshape(2, M).T.astype(np.float64), 128, 1)
    sb_diag = np.repeat(sB.reshape(2, 2).diagonal().astype(np.float64), 128)
    assert np.array_equal(got, decoded(A, True) * sa_full * sb_diag[None, :])


def test_gemm_rejects_unknown_format():
    A = np.zeros((4, 128), np.uint8)
    s = np.ones(4, np.float32)
    with pytest.raises(ValueError):
        oracle.gemm_rows(A, s, oracle.ROW, A, s, oracle.ROW, np.arange(4), fmtA=2)
