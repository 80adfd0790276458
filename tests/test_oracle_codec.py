"""Pins of the oracle's E4M3 codec (Q_FP8 of Eq. 3, paper Sec. 2.2) against
the OCP E4M3 definition, an independent encoder, brute force, and torch's
float8_e4m3fn conversion.  CPU only."""
import ctypes
import math
import os
import struct

import numpy as np
import pytest
import torch

import oracle

from _cbuild import helper

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "e4m3_key_values.txt")


def f32(bits):
    return struct.unpack("<f", struct.pack("<I", bits))[0]


def torch_decode_all():
    codes = torch.arange(256, dtype=torch.int32).to(torch.uint8)
    return codes.view(torch.float8_e4m3fn).to(torch.float64).numpy()


def test_golden_key_values():
    with open(GOLDEN) as fh:
        rows = [ln.split("#")[0].split() for ln in fh if ln.strip() and not ln.startswith("#")]
    assert len(rows) == 10
    for code_hex, val in rows:
        got = oracle.decode(int(code_hex, 16))
        if val == "nan":
            assert math.isnan(got)
        else:
            want = float(val)
            assert got == want and math.copysign(1, got) == math.copysign(1, want), code_hex


def test_decode_all_256_matches_torch():
    ref = torch_decode_all()
    for c in range(256):
        got = oracle.decode(c)
        if math.isnan(ref[c]):
            assert math.isnan(got), c
        else:
            assert got == ref[c], (c, got, ref[c])
            assert math.copysign(1, got) == math.copysign(1, ref[c])
    assert sum(math.isnan(oracle.decode(c)) for c in range(256)) == 2


def test_decode_monotone_and_distinct():
    vals = [oracle.decode(c) for c in range(0x7F)]
    assert all(a < b for a, b in zip(vals, vals[1:]))
    assert len(set(vals)) == 127
    assert vals[-1] == 448.0 and vals[1] == 2.0 ** -9 and vals[8] == 2.0 ** -6
    for c in range(0x7F):
        assert oracle.decode(c | 0x80) == -vals[c]


def test_encode_decode_roundtrip_254_codes():
    for c in range(256):
        if c in (0x7F, 0xFF):
            continue
        v = oracle.decode(c)
        assert oracle.encode(v) == c, hex(c)
    assert oracle.encode(-0.0) == 0x80 and oracle.encode(0.0) == 0x00


def test_midpoints_ties_to_even_and_neighbours():
    vals = [oracle.decode(c) for c in range(0x7F)]
    for c in range(0x7E):
        lo, hi = vals[c], vals[c + 1]
        mid = np.float32((lo + hi) / 2)
        assert float(mid) == (lo + hi) / 2  # exact in fp32
        even = c if c % 2 == 0 else c + 1
        assert oracle.encode(float(mid)) == even, hex(c)
        assert oracle.encode(-float(mid)) == even | 0x80
        up = np.nextafter(mid, np.float32(np.inf), dtype=np.float32)
        dn = np.nextafter(mid, np.float32(0), dtype=np.float32)
        assert oracle.encode(float(up)) == c + 1
        assert oracle.encode(float(dn)) == c
        assert oracle.encode(-float(up)) == (c + 1) | 0x80
        assert oracle.encode(-float(dn)) == c | 0x80


def test_saturation():
    for v in [448.0, 448.5, 455.0, 463.99, 464.0, 464.01, 480.0, 1e4,
              3.0e38, f32(0x7F7FFFFF), math.inf]:
        assert oracle.encode(v) == 0x7E, v
        assert oracle.encode(-v) == 0xFE, v


def test_exhaustive_against_independent_encoder():
    """Every fp32 pattern whose magnitude lies in [2^-12, 2^10) (where the
    encoding is not trivially 0 or 448), plus every 97th pattern elsewhere;
    set FP8_FULL_SWEEP=1 to walk all 2^32 patterns."""
    lib = helper("e4m3_sweep", link_oracle=True)
    lib.sweep.argtypes = [ctypes.c_uint64, ctypes.c_uint64, ctypes.c_uint64,
                          ctypes.c_int, ctypes.POINTER(ctypes.c_uint64),
                          ctypes.POINTER(ctypes.c_uint32)]
    lib.sweep.restype = ctypes.c_uint64
    threads = min(16, len(os.sched_getaffinity(0)))
    checked, first = ctypes.c_uint64(), ctypes.c_uint32()

    def run(start, end, stride):
        bad = lib.sweep(start, end, stride, threads, ctypes.byref(checked),
                        ctypes.byref(first))
        assert bad == 0, "mismatch at 0x%08x" % first.value
        return checked.value

    if os.environ.get("FP8_FULL_SWEEP") == "1":
        assert run(0, 1 << 32, 1) == (1 << 32) - 2 * ((1 << 23) - 1)
        return
    lo, hi = (127 - 12) << 23, (127 + 10) << 23
    n = 0
    for sign in (0, 1 << 31):
        n += run(sign | lo, sign | hi, 1)
        n += run(sign, sign | lo, 97)
        n += run(sign | hi, sign | 0x7FFFFFFF, 97)
    assert n > 2 * (hi - lo)


def brute_force(v, table):
    """Nearest member of the value table by exhaustive scan; ties to the even
    code; |v| >= 448 clamps."""
    a = abs(v)
    sign = 0x80 if math.copysign(1, v) < 0 else 0
    if a >= 448:
        return sign | 0x7E
    best, bestd = None, None
    for c, t in enumerate(table):
        d = abs(a - t)
        if bestd is None or d < bestd or (d == bestd and c % 2 == 0):
            best, bestd = c, d
    return sign | best


def test_brute_force_sample():
    table = [oracle.decode(c) for c in range(0x7F)]
    rng = np.random.default_rng(7)
    bits = rng.integers(0, 1 << 32, size=4000, dtype=np.uint64).astype(np.uint32)
    vals = [f32(int(b)) for b in bits]
    # concentrate on the interesting range as well
    vals += list(rng.uniform(-500, 500, 3000)) + list(rng.uniform(-0.02, 0.02, 3000))
    for v in vals:
        v = float(np.float32(v))
        if math.isnan(v):
            continue
        assert oracle.encode(v) == brute_force(v, table), v


def test_matches_torch_cast_in_range():
    """torch's float8_e4m3fn conversion rounds to nearest even and is only
    compared where it does not need saturation (|v| <= 464)."""
    rng = np.random.default_rng(11)
    x = np.concatenate([
        rng.standard_normal(200000).astype(np.float32) * 100,
        rng.standard_normal(200000).astype(np.float32) * 1e-3,
        rng.uniform(-464, 464, 200000).astype(np.float32),
    ])
    x = x[np.abs(x) <= 464]
    want = torch.from_numpy(x).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    got = oracle.cast_f32(x, 1.0)
    assert np.array_equal(got, want)
