"""The GEMM's scale-vector loads stay inside the scale arrays: a host model
of the per-lane offsets that paper_2609_22870_amd/csrc/gemm.hip forms in
gemm_tile's scale_offsets() and load_scales() (voffset per lane, soffset =
base + K block x stride), evaluated for every tile of ragged problems, every
K block, every tile shape and every blockwise pair, and for the sub-problems
of a split launch (scale arrays re-based at the split row or column, their
strides those of the whole problem).  Lanes whose offset is the out-of-range
marker (the weight-block lanes past the tile's blocks) are the only ones
allowed past the array; every other address must lie inside it, whatever
the hardware's range check covers.  No GPU is involved."""
import itertools

import pytest

OUT = 0x7fffffff                       # offset past any buffer: the load reads zero
TILES = [(256, 256, 8), (128, 128, 4), (128, 128, 8), (64, 64, 4)]   # BM, BN, waves of a K group


def scale_loads(pair, BM, BN, waves, M, N, K, m0, n0, sa_ld, sb_ld):
    """(array, byte offset) of every lane's load of every K block for the
    tile at (m0, n0); array None for marker lanes."""
    kblocks = K // 128
    kScaleA = BM * 4
    kScaleB = BN * 4 if pair == "blockk" else 256
    kQA, kQB = kScaleA // 256, kScaleB // 256
    assert kQA + kQB <= waves
    last_m, last_n = M - 1 - m0, N - 1 - n0
    out = []
    for wave in range(kQA + kQB):
        for lane in range(64):
            if wave < kQA:
                r = wave * 64 + lane
                voff, ld, base, arr = min(r, last_m) * 4, sa_ld * 4, m0 * 4, "A"
            elif pair == "block":
                nb = n0 // 128 + min(lane, last_n // 128)
                voff = nb * kblocks * 4 if lane < (BN + 127) // 128 else OUT
                ld, base, arr = 4, 0, "B"
            else:
                c = (wave - kQA) * 64 + lane
                voff, ld, base, arr = min(c, last_n) * 4, sb_ld * 4, n0 * 4, "B"
            for kt in range(kblocks):
                out.append((None if voff == OUT else arr, base + kt * ld + voff))
    return out


def check_problem(pair, BM, BN, waves, M, N, K, sa_ld, sb_ld, sa_count, sb_count):
    worst = {"A": -1, "B": -1}
    for tm, tn in itertools.product(range((M + BM - 1) // BM), range((N + BN - 1) // BN)):
        for arr, off in scale_loads(pair, BM, BN, waves, M, N, K, tm * BM, tn * BN, sa_ld, sb_ld):
            if arr is not None:
                worst[arr] = max(worst[arr], off + 4)
    assert 0 < worst["A"] <= sa_count * 4, (pair, BM, BN, M, N, K, worst, sa_count)
    assert 0 < worst["B"] <= sb_count * 4, (pair, BM, BN, M, N, K, worst, sb_count)


@pytest.mark.parametrize("BM,BN,waves", TILES)
@pytest.mark.parametrize("pair", ["block", "blockk"])
@pytest.mark.parametrize("M,N,K", [(272, 384, 640), (1, 128, 128), (300, 256, 256), (129, 512, 384)])
def test_scale_loads_in_bounds(pair, BM, BN, waves, M, N, K):
    if pair == "blockk":
        N = N + 4                       # per-column scales: any N
    kb = K // 128
    sa_count = kb * M                   # 1x128: [K/128][M]
    sb_count = kb * N if pair == "blockk" else (N // 128) * kb   # [K/128][N] or [N/128][K/128]
    check_problem(pair, BM, BN, waves, M, N, K, M, N, sa_count, sb_count)


@pytest.mark.parametrize("pair", ["block", "blockk"])
def test_scale_loads_in_bounds_split_launch(pair):
    """Sub-problems of a split launch: rows [m, m + Ms) and columns [n, n +
    Ns) of the whole problem, scale arrays re-based at m (A) and at n or its
    weight block (B), strides those of the whole problem, counts the rest of
    the arrays."""
    M, N, K = 700, 1280 if pair == "block" else 1292, 256
    kb = K // 128
    for (m, Ms), (n, Ns) in itertools.product([(0, 512), (512, M - 512)], [(0, 1024), (1024, N - 1024)]):
        if pair == "block":
            sb_count = (N // 128) * kb - (n // 128) * kb
        else:
            sb_count = kb * N - n
        for BM, BN, waves in TILES:
            check_problem(pair, BM, BN, waves, Ms, Ns, K, M, N, kb * M - m, sb_count)
