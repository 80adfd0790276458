"""Pins of the oracle quantizer: Eq. 3 (paper Sec. 2.2) per scaling unit at
tensorwise, rowwise and blockwise granularity.  CPU only.

The pins are invariants of the definition (granularities that must coincide,
power-of-two scale invariance, the dequantization error bound), special
cases with known codes, and a reference built from torch library routines
(amax by reshaping into units, fp32 division, torch's float8_e4m3fn cast)."""
import math

import numpy as np
import pytest
import torch

import oracle
from paper_2609_22870_amd import synth

G_ALL = [oracle.TENSOR, oracle.ROW, oracle.COL, oracle.BLOCK_1x128,
         oracle.BLOCK_128x1, oracle.BLOCK_128x128]
G_T = {oracle.ROW: oracle.COL, oracle.COL: oracle.ROW,
       oracle.BLOCK_1x128: oracle.BLOCK_128x1, oracle.BLOCK_128x1: oracle.BLOCK_1x128}


def bits(t):
    return synth.bf16_bits(t)


def torch_reference(x, g):
    """Codes and scales by torch routines, units cut out by reshaping.
    Scale layouts as documented for the oracle (not transposed)."""
    xf = x.float()
    R, C = xf.shape
    if g == oracle.TENSOR:
        units = xf.reshape(1, 1, R * C)
    elif g == oracle.ROW:
        units = xf.reshape(R, 1, C)
    elif g == oracle.COL:
        units = xf.t().reshape(C, 1, R)
    elif g == oracle.BLOCK_1x128:
        units = xf.reshape(R, C // 128, 128).permute(1, 0, 2)  # [kb, r, 128]
    elif g == oracle.BLOCK_128x1:
        units = xf.reshape(R // 128, 128, C).permute(0, 2, 1)  # [rb, c, 128]
    else:
        units = xf.reshape(R // 128, 128, C // 128, 128).permute(0, 2, 1, 3)
        units = units.reshape(R // 128, C // 128, 128 * 128)
    amax = units.abs().amax(dim=-1, keepdim=True)
    s = amax / 448.0
    s = torch.where(s == 0, torch.ones_like(s), s)
    q = (units / s).to(torch.float8_e4m3fn).view(torch.uint8)
    # put codes back in matrix order
    if g == oracle.TENSOR:
        codes = q.reshape(R, C)
    elif g == oracle.ROW:
        codes = q.reshape(R, C)
    elif g == oracle.COL:
        codes = q.reshape(C, R).t()
    elif g == oracle.BLOCK_1x128:
        codes = q.permute(1, 0, 2).reshape(R, C)
    elif g == oracle.BLOCK_128x1:
        codes = q.permute(0, 2, 1).reshape(R, C)
    else:
        codes = q.reshape(R // 128, C // 128, 128, 128).permute(0, 2, 1, 3).reshape(R, C)
    return codes.contiguous().numpy(), s.reshape(-1).numpy()


def sample(rows, cols, seed, outliers=True):
    ocols = synth.outlier_columns(cols, seed + 1) if outliers else None
    return synth.normal_bf16((rows, cols), 1.0, seed, outlier_cols=ocols)


@pytest.mark.parametrize("g", G_ALL)
def test_matches_torch_reference(g):
    x = sample(256, 384, 3)
    codes, scales = oracle.quantize(bits(x), g)
    rc, rs = torch_reference(x, g)
    assert np.array_equal(scales, rs)
    assert np.array_equal(codes, rc)


@pytest.mark.parametrize("g", G_ALL)
def test_transposed_output_is_quantization_of_transpose(g):
    x = sample(256, 384, 5)
    codes, scales = oracle.quantize(bits(x), g, transposed=True)
    c2, s2 = oracle.quantize(bits(x.t().contiguous()), G_T.get(g, g))
    assert codes.shape == (384, 256)
    assert np.array_equal(codes, c2) and np.array_equal(scales, s2)
    # and the codes are the byte transpose of the plain mode
    c3, _ = oracle.quantize(bits(x), g)
    assert np.array_equal(codes, c3.T)


def plant_max(x, g, value):
    """Make every unit of granularity g hold `value` as its largest magnitude:
    clip everything to below it and write +-value at one position per unit."""
    x = x.float().clamp(-value / 2, value / 2)
    R, C = x.shape
    rng = np.random.default_rng(0)
    if g == oracle.ROW:
        for r in range(R):
            x[r, rng.integers(C)] = value * (1 if r % 2 else -1)
    elif g == oracle.BLOCK_1x128:
        for r in range(R):
            for kb in range(C // 128):
                x[r, kb * 128 + rng.integers(128)] = -value
    elif g == oracle.BLOCK_128x1:
        for c in range(C):
            for rb in range(R // 128):
                x[rb * 128 + rng.integers(128), c] = value
    elif g == oracle.BLOCK_128x128:
        for rb in range(R // 128):
            for cb in range(C // 128):
                x[rb * 128 + rng.integers(128), cb * 128 + rng.integers(128)] = value
    return x.to(torch.bfloat16)


@pytest.mark.parametrize("g", [oracle.ROW, oracle.BLOCK_1x128, oracle.BLOCK_128x1,
                               oracle.BLOCK_128x128])
def test_equals_tensorwise_when_every_unit_amax_matches(g):
    x = plant_max(sample(256, 256, 9, outliers=False), g, 3.0)
    codes, scales = oracle.quantize(bits(x), g)
    tcodes, tscale = oracle.quantize(bits(x), oracle.TENSOR)
    assert np.array_equal(codes, tcodes)
    assert np.all(scales == tscale[0])


def test_granularities_that_coincide():
    x = sample(128, 128, 13)
    b = bits(x)
    row = oracle.quantize(b, oracle.ROW)
    blk = oracle.quantize(b, oracle.BLOCK_1x128)
    assert np.array_equal(row[0], blk[0]) and np.array_equal(row[1], blk[1])
    col = oracle.quantize(b, oracle.COL)
    blk = oracle.quantize(b, oracle.BLOCK_128x1)
    assert np.array_equal(col[0], blk[0]) and np.array_equal(col[1], blk[1])
    ten = oracle.quantize(b, oracle.TENSOR)
    blk = oracle.quantize(b, oracle.BLOCK_128x128)
    assert np.array_equal(ten[0], blk[0]) and np.array_equal(ten[1], blk[1])
    # cols = 128 but more rows: 1x128 is still rowwise
    x = sample(384, 128, 14)
    row = oracle.quantize(bits(x), oracle.ROW)
    blk = oracle.quantize(bits(x), oracle.BLOCK_1x128)
    assert np.array_equal(row[0], blk[0]) and np.array_equal(row[1], blk[1])


@pytest.mark.parametrize("g", G_ALL)
@pytest.mark.parametrize("j", [-40, -3, 9])
def test_power_of_two_scale_invariance(g, j):
    x = sample(256, 256, 17)
    y = (x.float() * 2.0 ** j).to(torch.bfloat16)
    assert torch.equal(y.float(), x.float() * 2.0 ** j)  # exact in bf16
    cx, sx = oracle.quantize(bits(x), g)
    cy, sy = oracle.quantize(bits(y), g)
    assert np.array_equal(cx, cy)
    assert np.array_equal(sy, (sx.astype(np.float64) * 2.0 ** j).astype(np.float32))


@pytest.mark.parametrize("g", G_ALL)
def test_dequantization_error_bound(g):
    x = sample(256, 256, 19)
    codes, scales = oracle.quantize(bits(x), g)
    table = np.array([oracle.decode(c) if c not in (0x7F, 0xFF) else np.nan
                      for c in range(256)])
    dec = table[codes]
    _, s_full = expand_scales(x, g)
    xf = x.float().numpy().astype(np.float64)
    err = np.abs(xf - s_full * dec)
    q = xf / s_full
    bound = s_full * (np.maximum(2.0 ** -4 * np.abs(dec), 2.0 ** -10) + 2.0 ** -23 * np.abs(q))
    assert np.all(err <= bound)
    assert np.all(np.abs(dec) <= 448)


def expand_scales(x, g):
    """Scale of every element, from torch_reference's unit geometry."""
    xf = x.float()
    R, C = xf.shape
    _, s = torch_reference(x, g)
    if g == oracle.TENSOR:
        full = np.full((R, C), s[0])
    elif g == oracle.ROW:
        full = np.repeat(s[:, None], C, axis=1)
    elif g == oracle.COL:
        full = np.repeat(s[None, :], R, axis=0)
    elif g == oracle.BLOCK_1x128:
        full = np.repeat(s.reshape(C // 128, R).T, 128, axis=1)
    elif g == oracle.BLOCK_128x1:
        full = np.repeat(s.reshape(R // 128, C), 128, axis=0)
    else:
        full = np.repeat(np.repeat(s.reshape(R // 128, C // 128), 128, 0), 128, 1)
    return s, full.astype(np.float64)


def block(values):
    """A 1 x 128 bf16 row from python floats (must be bf16-exact)."""
    t = torch.tensor(values, dtype=torch.float32)
    b = t.to(torch.bfloat16)
    assert torch.equal(b.float(), t)
    return b.reshape(1, -1)


def test_single_nonzero_block():
    for v in [1.0, -3.5, 1e-3, 2.0 ** -130, 6.0e37]:
        v = float(torch.tensor(v).to(torch.bfloat16).float())
        vals = [0.0] * 128
        vals[77] = v
        codes, scales = oracle.quantize(bits(block(vals)), oracle.BLOCK_1x128)
        assert scales[0] == np.float32(np.float32(abs(v)) / np.float32(448.0))
        assert codes[0, 77] == (0xFE if v < 0 else 0x7E)
        assert np.all(np.delete(codes[0], 77) == 0)


def test_constant_magnitude_block():
    vals = [0.75 if i % 3 else -0.75 for i in range(128)]
    codes, scales = oracle.quantize(bits(block(vals)), oracle.BLOCK_1x128)
    assert scales[0] == np.float32(0.75) / np.float32(448)
    assert np.array_equal(codes[0], np.where(np.array(vals) < 0, 0xFE, 0x7E))


def test_all_zero_block():
    vals = [0.0] * 64 + [-0.0] * 64
    codes, scales = oracle.quantize(bits(block(vals)), oracle.BLOCK_1x128)
    assert scales[0] == 1.0
    assert np.all(codes[0, :64] == 0x00) and np.all(codes[0, 64:] == 0x80)


def test_subnormal_amax_block():
    # bf16 subnormals: the scale is an fp32 subnormal; without flush to zero
    # the largest element still maps to 448.
    vals = [2.0 ** -133 * (i % 5) for i in range(127)] + [-(2.0 ** -128)]
    codes, scales = oracle.quantize(bits(block(vals)), oracle.BLOCK_1x128)
    assert 0 < scales[0] < np.finfo(np.float32).tiny
    assert codes[0, 127] == 0xFE


def test_amax_element_always_encodes_to_448():
    """For every positive finite bf16 amax a, the element equal to a encodes
    to 0x7E (RN32(a / RN32(a / 448)) stays within the rounding range of 448)."""
    a = np.arange(1, 0x7F80, dtype=np.uint16)  # all positive finite bf16
    x = np.zeros((a.size, 128), dtype=np.uint16)
    x[:, 5] = a
    x[:, 6] = a | 0x8000
    codes, _ = oracle.quantize(x, oracle.ROW)
    assert np.all(codes[:, 5] == 0x7E) and np.all(codes[:, 6] == 0xFE)


def test_ties_through_the_whole_path():
    """A block whose amax is 448 * 2^k has S = 2^k exactly, so x / S is exact
    and midpoints between E4M3 neighbours must go to the even code."""
    table = [oracle.decode(c) for c in range(0x7F)]
    mids = [(table[c] + table[c + 1]) / 2 for c in range(0x7E)]
    want = [c if c % 2 == 0 else c + 1 for c in range(0x7E)]
    for k in (-20, 0, 5):
        vals = [m * 2.0 ** k for m in mids] + [448.0 * 2.0 ** k]
        vals += [-v for v in vals[: 128 - len(vals)]]
        vals = vals[:128]
        codes, scales = oracle.quantize(bits(block(vals)), oracle.BLOCK_1x128)
        assert scales[0] == 2.0 ** k
        assert list(codes[0, :0x7E]) == want
        assert codes[0, 0x7E] == 0x7E
        assert list(codes[0, 0x7F:]) == [w | 0x80 for w in want[: 128 - 0x7F]]


def test_rejects_bad_shapes():
    x = np.zeros((100, 256), dtype=np.uint16)
    with pytest.raises(ValueError):
        oracle.quantize(x, oracle.BLOCK_128x1)
    with pytest.raises(ValueError):
        oracle.quantize(x, oracle.BLOCK_128x128)
    with pytest.raises(ValueError):
        oracle.quantize(np.zeros((128, 200), dtype=np.uint16), oracle.BLOCK_1x128)
    oracle.quantize(x, oracle.BLOCK_1x128)  # fine: cols multiple of 128


def test_division_not_reciprocal():
    """Eq. 3 divides by S.  For some bf16 pairs (amax, x) the quotient
    RN32(x / S) and the product RN32(x * RN32(1 / S)) fall on opposite sides
    of an E4M3 rounding boundary; the oracle must follow the division
    (computed here by torch in fp32) on every such pair in amax in [1, 8)."""
    allx = (np.arange(1, 0x7F80, dtype=np.uint32) << 16).view(np.float32)
    found = 0
    for ai in range(0x3F80, 0x4100):
        a = (np.array([ai], dtype=np.uint32) << 16).view(np.float32)[0]
        S = np.float32(a / np.float32(448))
        xs = allx[allx <= a]
        q_div = torch.from_numpy(xs) / torch.tensor(S)
        q_rcp = torch.from_numpy(xs) * (torch.tensor(np.float32(1)) / torch.tensor(S))
        c_div = q_div.to(torch.float8_e4m3fn).view(torch.uint8).numpy()
        c_rcp = q_rcp.to(torch.float8_e4m3fn).view(torch.uint8).numpy()
        diff = np.nonzero(c_div != c_rcp)[0]
        if diff.size == 0:
            continue
        found += diff.size
        x = np.zeros((1, 128), dtype=np.uint16)
        x[0, 0] = ai
        sel = xs[diff[:127]].view(np.uint32) >> 16
        x[0, 1:1 + sel.size] = sel
        codes, scales = oracle.quantize(x, oracle.BLOCK_1x128)
        assert scales[0] == S
        assert np.array_equal(codes[0, 1:1 + sel.size], c_div[diff[:127]])
    assert found > 50


# ---- the power-of-two scale variant (not the paper's scale): S is the
# smallest power of two with 448 S >= amax, at least 2^-127

def exact_pow2_scale(amax):
    """Smallest power of two S (as a Fraction exponent search) with 448 S >=
    amax, clamped at 2^-127; 1 for amax = 0."""
    from fractions import Fraction
    a = Fraction(amax)
    if a == 0:
        return 1.0
    k = 0
    while 448 * Fraction(2) ** k < a:
        k += 1
    while 448 * Fraction(2) ** (k - 1) >= a:
        k -= 1
    return float(Fraction(2) ** max(k, -127))


def test_pow2_scales_against_exact_search():
    """Single-unit (tensorwise) quantizations of amaxes across the bf16
    range, including 448 * 2^k and its bf16 neighbours, subnormals and the
    largest finite bf16."""
    amaxes = [448.0 * 2.0 ** k for k in range(-20, 20)]
    amaxes += [float(torch.tensor(v, dtype=torch.float32).to(torch.bfloat16).float() * f)
               for v in (1.0, 3.0, 0.875, 0.9, 1.75, 1.7578125) for f in (1.0, 2.0 ** -60, 2.0 ** 70)]
    amaxes += [2.0 ** -133, 2.0 ** -130, 1.5 * 2.0 ** -127, 3.3895313892515355e38, 0.0]
    for amax in amaxes:
        x = torch.tensor([[amax, -amax / 4.0]], dtype=torch.float32).to(torch.bfloat16)
        a = float(x.float().abs().max())
        _, s = oracle.quantize(bits(x), oracle.TENSOR, pow2=True)
        assert float(s[0]) == exact_pow2_scale(a), (a, s[0])


@pytest.mark.parametrize("g", G_ALL)
def test_pow2_codes_are_exact_quotients(g):
    """S is a power of two, so x / S is exact: every code is the nearest
    E4M3 value of the exact quotient, no quotient exceeds 448, and the
    dequantization error is at most half a unit in the last place."""
    x = sample(256, 256, 23)
    codes, scales = oracle.quantize(bits(x), g, pow2=True)
    assert np.all(np.frexp(scales.astype(np.float64))[0] == 0.5)       # powers of two
    table = np.array([oracle.decode(c) if c not in (0x7F, 0xFF) else np.nan for c in range(256)])
    dec = table[codes]
    # the unit geometry of the fp32 mode, with the power-of-two scales
    s_plain, full_plain = expand_scales(x, g)
    full = np.zeros_like(full_plain)
    for v_plain, v_pow2 in zip(np.asarray(s_plain, dtype=np.float64), scales.astype(np.float64)):
        full[full_plain == v_plain] = v_pow2
    xf = x.float().numpy().astype(np.float64)
    q = xf / full
    assert np.all(np.abs(q) <= 448)
    assert np.all(np.abs(xf - full * dec) <= full * np.maximum(2.0 ** -4 * np.abs(dec), 2.0 ** -10))


def test_pow2_matches_plain_scale_when_amax_is_448_times_a_power_of_two():
    """amax = 448 * 2^j makes both scales 2^j: identical codes and scales."""
    x = sample(128, 256, 29, outliers=False)
    x = plant_max(x, oracle.BLOCK_1x128, 448.0 * 2.0 ** -9)
    c1, s1 = oracle.quantize(bits(x), oracle.BLOCK_1x128)
    c2, s2 = oracle.quantize(bits(x), oracle.BLOCK_1x128, pow2=True)
    assert np.array_equal(s1, s2) and np.array_equal(c1, c2)
