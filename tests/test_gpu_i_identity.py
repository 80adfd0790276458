"""The GEMM's exact special case (the bit-exact pin of the scaled GEMM of
Sec. 2.2's FP8 linear layer) on every tile kernel, on split launches, and in
every GEMM form.

B holds identity codes (1.0 where n == k, for the first N <= K indices) and
every scale is a power of two between 2^-6 and 2^6, so each output element
is one exact product: C[m][n] = S_A(m, kb) S_B(n, kb) decode(A[m][n]) with
kb = n / 128 the K block of that product.  Every partial sum, scale product,
promotion and rounding step on the way is exact (fp32 products of 4-bit
significands and powers of two; bf16 keeps 8 significant bits), so the
output must equal that value bit for bit (+0 and -0 compare equal: the sum
of the zero products has no defined sign).  A's codes are random finite
codes; they and the scales are inputs, so no FP8 quantization is involved
(the quantizers are pinned byte for byte elsewhere).

Shapes are chosen to reach each launch path: 256 x 256 tiles (at least 512
of them; N = 4096 spans two odd 1024-column bands, which walk K backwards),
128 x 128 tiles of four waves (at least 256 of them) and of eight waves
(128 to 255 of them), 64 x 64 tiles with two K groups (an even number of K
blocks on at most 256 tiles) and with one, and problems split into
sub-launches because an operand spans 2 GiB (along N, and along M).  The
scales vary per row, column and block (no two neighbouring blocks alike by
construction), so a scale read from the wrong row, column or K block
shows."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_22870_amd as fp8q
from paper_2609_22870_amd import synth

import _par

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
ONE = {False: 0x38, True: 0x3C}   # the code of 1.0 in E4M3, E5M2

_TABLES = {}


def table(e5m2):
    if e5m2 not in _TABLES:
        dec = oracle.decode_e5m2 if e5m2 else oracle.decode
        _TABLES[e5m2] = np.array([dec(c) for c in range(256)], dtype=np.float64)
    return _TABLES[e5m2]


def random_codes(M, K, seed, e5m2=False):
    """Finite codes: magnitude codes below the format's NaN / infinity
    codes, random sign."""
    g = torch.Generator(device=DEV)
    g.manual_seed(seed)
    mag = torch.randint(0, 0x7C if e5m2 else 0x7F, (M, K), generator=g, device=DEV, dtype=torch.uint8)
    sign = torch.randint(0, 2, (M, K), generator=g, device=DEV, dtype=torch.uint8) * 0x80
    return mag | sign


def pow2_scales(n, seed):
    rng = np.random.default_rng(seed)
    return (2.0 ** rng.integers(-6, 7, size=n)).astype(np.float32)


def identity(N, K, e5m2=False):
    B = torch.zeros((N, K), dtype=torch.uint8, device=DEV)
    idx = torch.arange(N, device=DEV)
    B[idx, idx] = ONE[e5m2]
    return B


def scale_count(rows, cols, g):
    return fp8q.scales_count(rows, cols, g)


def expected(A_cols, sa, ga, sb, gb, M, N, K, e5m2_a=False):
    """The exact output from A's first N columns (host codes [M, N]) and the
    host scale arrays in the layouts of fp8q_scales_count."""
    kb = np.arange(N) // 128
    dA = table(e5m2_a)[A_cols]
    if ga == fp8q.TENSOR:
        s_a = np.float64(sa[0])
    elif ga == fp8q.ROW:
        s_a = sa.astype(np.float64)[:, None]
    else:                                   # 1x128: [K/128][M]
        s_a = sa.reshape(K // 128, M).astype(np.float64)[kb, :].T
    if gb == fp8q.TENSOR:
        s_b = np.float64(sb[0])
    elif gb == fp8q.ROW:
        s_b = sb.astype(np.float64)[None, :]
    elif gb == fp8q.BLOCK_128x128:          # [N/128][K/128]
        s_b = sb.reshape(-1, K // 128).astype(np.float64)[np.arange(N) // 128, kb][None, :]
    else:                                   # 1x128: [K/128][N]
        s_b = sb.reshape(K // 128, N).astype(np.float64)[kb, np.arange(N)][None, :]
    want = dA * s_a * s_b
    w32 = want.astype(np.float32)
    assert np.array_equal(w32.astype(np.float64), want), "expected values must be exact in fp32"
    wb = torch.from_numpy(w32).to(torch.bfloat16)
    assert torch.equal(wb.float(), torch.from_numpy(w32)), "expected values must be exact in bf16"
    return wb


def check(got, want, label):
    bad = (got.float() != want.float()).nonzero()
    if bad.numel():
        for m, n in bad[:8].tolist():
            print("  %s: m=%d n=%d got=%r want=%r" % (label, m, n, got[m, n].item(), want[m, n].item()), flush=True)
    assert bad.numel() == 0, "%s: %d mismatches" % (label, bad.shape[0])


class Case:
    """A: random codes [M, K]; B: identity [N, K]; power-of-two scales."""

    def __init__(self, ga, gb, M, K, N, seed, e5m2_a=False, e5m2_b=False, share_a=None):
        assert N <= K
        self.ga, self.gb, self.M, self.K, self.N = ga, gb, M, K, N
        self.e5m2_a = e5m2_a
        if share_a is None:
            self.A = random_codes(M, K, seed, e5m2_a)
            self.sa = pow2_scales(scale_count(M, K, ga), seed + 1)
            self.sA = torch.from_numpy(self.sa).to(DEV)
        else:                               # another problem on the same A
            self.A, self.sa, self.sA = share_a.A, share_a.sa, share_a.sA
        self.B = identity(N, K, e5m2_b)
        self.sb = pow2_scales(scale_count(N, K, gb), seed + 2)
        self.sB = torch.from_numpy(self.sb).to(DEV)

    def want(self):
        a_cols = self.A[:, :self.N].cpu().numpy()
        return expected(a_cols, self.sa, self.ga, self.sb, self.gb, self.M, self.N, self.K, self.e5m2_a)


PAIRS = {
    "tensor": (fp8q.TENSOR, fp8q.TENSOR),
    "row": (fp8q.ROW, fp8q.ROW),
    "block": (fp8q.BLOCK_1x128, fp8q.BLOCK_128x128),
    "blockk": (fp8q.BLOCK_1x128, fp8q.BLOCK_1x128),
}
# (M, K, N): the launch path each reaches
# (the (1x128, 1x128) pair has no 256 x 256 kernel: on the first shape it
# runs its 128 x 128 kernel over many tiles)
SHAPES = {
    "256x256 tiles": (8192 + 96, 4096, 4096),     # 33 x 16 = 528 big tiles, ragged last tile row
    "128x128 tiles": (4096 + 32, 1024, 1024),     # 33 x 8 = 264 mid tiles, 68 big ones
    "128x128 eight-wave tiles": (256 + 32, 6144, 6144),  # 3 x 48 = 144 mid tiles, 4 K bands
    "64x64 two K groups": (160, 512, 512),        # 3 x 8 tiles, 4 K blocks
    "64x64 one K group": (160, 384, 384),         # 3 K blocks
}


@pytest.mark.parametrize("shape", list(SHAPES))
@pytest.mark.parametrize("pair", list(PAIRS))
def test_identity_every_kernel(pair, shape):
    ga, gb = PAIRS[pair]
    M, K, N = SHAPES[shape]
    print("identity pin", pair, shape, (M, K, N), flush=True)
    c = Case(ga, gb, M, K, N, seed=1000 + 17 * list(PAIRS).index(pair) + list(SHAPES).index(shape))
    C = fp8q.gemm(c.A, c.sA, ga, c.B, c.sB, gb)
    torch.cuda.synchronize()
    check(C.cpu(), c.want(), "%s %s" % (pair, shape))


@pytest.mark.parametrize("pair", ["tensor", "row", "block", "blockk"])
def test_identity_split_along_n(pair):
    """B spans more than 2 GiB (N = K = 46464): two sub-launches along N,
    the first on 256 x 256 tiles (or 128 x 128), the second on 128 x 128
    ones; B's scales are re-based at the split column."""
    ga, gb = PAIRS[pair]
    M, K, N = 2048 + 64, 46464, 46464
    print("identity pin split along N", pair, (M, K, N), flush=True)
    c = Case(ga, gb, M, K, N, seed=2000 + list(PAIRS).index(pair))
    C = fp8q.gemm(c.A, c.sA, ga, c.B, c.sB, gb)
    torch.cuda.synchronize()
    want = c.want()
    del c
    check(C.cpu(), want, "split N " + pair)


@pytest.mark.parametrize("pair", ["row", "block", "blockk"])
def test_identity_split_along_m(pair):
    """A spans more than 2 GiB (M = 46432 rows of K = 46464): two
    sub-launches along M (46080 rows on 256 x 256 tiles, then 352 rows), A's
    scales re-based at the split row."""
    ga, gb = PAIRS[pair]
    M, K, N = 46432, 46464, 768
    print("identity pin split along M", pair, (M, K, N), flush=True)
    c = Case(ga, gb, M, K, N, seed=3000 + list(PAIRS).index(pair))
    C = fp8q.gemm(c.A, c.sA, ga, c.B, c.sB, gb)
    torch.cuda.synchronize()
    want = c.want()
    del c
    check(C.cpu(), want, "split M " + pair)


@pytest.mark.parametrize("shape", list(SHAPES))
def test_identity_pow2_gemm(shape):
    """fp8q_gemm_pow2: the block scales enter the matrix instruction as
    exponents."""
    M, K, N = SHAPES[shape]
    print("identity pin pow2", shape, flush=True)
    c = Case(fp8q.BLOCK_1x128, fp8q.BLOCK_128x128, M, K, N, seed=4000 + list(SHAPES).index(shape))
    C = fp8q.gemm_pow2(c.A, c.sA, fp8q.BLOCK_1x128, c.B, c.sB, fp8q.BLOCK_128x128)
    torch.cuda.synchronize()
    check(C.cpu(), c.want(), "pow2 " + shape)


@pytest.mark.parametrize("formats", [fp8q.A_E5M2, fp8q.B_E5M2, fp8q.A_E5M2 | fp8q.B_E5M2])
@pytest.mark.parametrize("pair", ["block", "blockk"])
@pytest.mark.parametrize("shape", ["256x256 tiles", "128x128 tiles", "128x128 eight-wave tiles",
                                   "64x64 two K groups"])
def test_identity_e5m2_formats(pair, formats, shape):
    ga, gb = PAIRS[pair]
    M, K, N = SHAPES[shape]
    print("identity pin formats", pair, formats, shape, flush=True)
    c = Case(ga, gb, M, K, N, seed=5000 + 7 * formats + list(SHAPES).index(shape),
             e5m2_a=bool(formats & fp8q.A_E5M2), e5m2_b=bool(formats & fp8q.B_E5M2))
    C = fp8q.gemm_formats(c.A, c.sA, ga, c.B, c.sB, gb, formats)
    torch.cuda.synchronize()
    check(C.cpu(), c.want(), "formats %d %s %s" % (formats, pair, shape))


@pytest.mark.parametrize("pair", ["tensor", "row", "block"])
@pytest.mark.parametrize("ns,M", [((4096, 1024, 2048), 8192 + 96),    # 924 big tiles: 256 x 256
                                  ((1024, 512), 4096 + 32),            # 396 mid tiles: 128 x 128
                                  ((256, 512, 128), 160)])             # 64 x 64, K groups
def test_identity_grouped(pair, ns, M):
    """One launch over problems that share A (and K), each with its own
    identity B of N_i rows and its own scales."""
    ga, gb = PAIRS[pair]
    K = max(ns)
    print("identity pin grouped", pair, ns, M, flush=True)
    seed = 6000 + 31 * list(PAIRS).index(pair) + M
    base = Case(ga, gb, M, K, ns[0], seed=seed)
    cases = [base] + [Case(ga, gb, M, K, n, seed=seed + 10 * (i + 1), share_a=base) for i, n in enumerate(ns[1:])]
    outs = fp8q.gemm_grouped([(c.A, c.sA, c.B, c.sB) for c in cases], ga, gb)
    torch.cuda.synchronize()
    for i, (c, C) in enumerate(zip(cases, outs)):
        check(C.cpu(), c.want(), "grouped %s problem %d" % (pair, i))


@pytest.mark.parametrize("shape", ["256x256 tiles", "128x128 tiles"])
def test_identity_quantized_output(shape):
    """fp8q_gemm_quantized: the exact bf16 output, quantized per 1x128 unit
    along N by the oracle, must come out byte for byte."""
    M, K, N = SHAPES[shape]
    print("identity pin quantized output", shape, flush=True)
    c = Case(fp8q.BLOCK_1x128, fp8q.BLOCK_128x128, M, K, N, seed=7000 + list(SHAPES).index(shape))
    codes, scales = fp8q.gemm_quantized(c.A, c.sA, fp8q.BLOCK_1x128, c.B, c.sB, fp8q.BLOCK_128x128)
    torch.cuda.synchronize()
    want = c.want()
    oq, osq = _par.quantize(synth.bf16_bits(want), oracle.BLOCK_1x128)
    got_q = codes.cpu().numpy()
    # a zero output is a sum of zero products, whose sign is not defined:
    # its code may be 0x00 or 0x80
    bad = np.argwhere(np.where(got_q == 0x80, 0, got_q) != np.where(oq == 0x80, 0, oq))
    assert bad.shape[0] == 0, "%d code mismatches, first %s" % (bad.shape[0], bad[:4].tolist())
    assert np.array_equal(scales.cpu().numpy().view(np.uint32), osq.view(np.uint32))
