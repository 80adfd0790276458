"""The GEMM's workgroup-to-tile mapping: a host model of xcd_order() and
raster() in paper_2609_22870_amd/csrc/gemm.hip (workgroup b runs on XCD
b % 8 and takes position xcd_order(b) of the raster; the raster walks groups
of 8 tile rows, or of 8 tile columns when B is the larger operand and the two
together overflow the 256 MB last-level cache).  Every launch must cover each
tile of C exactly once; the mapping never changes an output element's K
order, which depends on its column alone.  No GPU is involved."""
import pytest

GROUP = 8
LLC = 256 << 20


def xcd_order(total, b):
    xcd, per, extra = b & 7, total >> 3, total & 7
    return xcd * per + min(xcd, extra) + (b >> 3)


def col_groups(M, N, K, BM):
    tiles_m = -(-M // BM)
    return N > M and tiles_m > GROUP and (M + N) * K > LLC


def raster(M, N, K, BM, BN, pos):
    tiles_m, tiles_n = -(-M // BM), -(-N // BN)
    cg = col_groups(M, N, K, BM)
    grouped, walked = (tiles_n, tiles_m) if cg else (tiles_m, tiles_n)
    per_group = GROUP * walked
    group = pos // per_group
    first = group * GROUP
    gsize = min(grouped - first, GROUP)
    in_group = pos - group * per_group
    across, along = first + in_group % gsize, in_group // gsize
    return (along, across) if cg else (across, along)


SHAPES = [  # (M, K, N, tile)
    (5120, 16384, 25600, 128),    # 32B up-projection wgrad: column groups
    (25600, 16384, 5120, 128),    # 32B down-projection wgrad
    (16384, 4096, 12288, 256),    # 8B up-projection forward
    (16384, 5120, 25600, 256),    # 32B up forward: operands fit the cache
    (16384, 25600, 5120, 256),
    (1152, 65536, 4096, 128),     # column groups, ragged group of tile columns
    (1100, 65536, 4100, 128),     # ragged tiles both ways
    (256, 12288, 4096, 64),       # decode: every tile row in one group
    (1, 128, 128, 64),
]


@pytest.mark.parametrize("M,K,N,T", SHAPES)
def test_every_tile_once(M, K, N, T):
    tiles_m, tiles_n = -(-M // T), -(-N // T)
    total = tiles_m * tiles_n
    seen = set()
    for b in range(total):
        tm, tn = raster(M, N, K, T, T, xcd_order(total, b))
        assert 0 <= tm < tiles_m and 0 <= tn < tiles_n
        seen.add((tm, tn))
    assert len(seen) == total


def test_orientation_of_the_named_layers():
    """Only the 32B up-projection's weight gradient (A = X^T 84 MB, B = dY^T
    419 MB) takes column groups among the named layer shapes."""
    assert col_groups(5120, 25600, 16384, 128)
    for M, K, N, T in [(25600, 16384, 5120, 128), (16384, 4096, 12288, 256), (16384, 12288, 4096, 256),
                       (16384, 4096, 6144, 256), (16384, 5120, 25600, 256), (16384, 25600, 5120, 256),
                       (256, 4096, 12288, 128), (256, 12288, 4096, 64)]:
        assert not col_groups(M, N, K, T), (M, K, N)


def test_xcd_shares_operand_bands():
    """The tiles one XCD runs together (its first 64 positions with two
    128 x 128 workgroups per CU) span 8 tile rows or 8 tile columns."""
    for M, K, N in [(5120, 16384, 25600), (25600, 16384, 5120)]:
        T = 128
        total = -(-M // T) * -(-N // T)
        first = [raster(M, N, K, T, T, xcd_order(total, b)) for b in range(0, 8 * 64, 8)]   # XCD 0
        rows, cols = {t[0] for t in first}, {t[1] for t in first}
        assert len(rows) == 8 and len(cols) == 8, (M, N, len(rows), len(cols))
