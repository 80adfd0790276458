"""GPU tests of fp8q_gemm_splitk, the split-K GEMM for skinny problems (a
decode step of the FP8 rollout: a few hundred activation rows against a
whole weight).  Each 128 x 128 tile's K blocks are split over S workgroups
whose fp32 partial tiles are added in split order by the last to arrive.

* Parity against the oracle at the 8B decode down-projection (256 x 12288 x
  4096, S = 4) and at small ragged shapes reaching S = 2, 4 and 8, for every
  pair, to the bar of the other GEMM tests (tests/_par.py check_gemm, with
  S - 1 more fp32 additions in the elementwise bound).
* The exact identity pin (test_gpu_i_identity's construction: each output
  one exact product) through every split count: the partial sums and their
  sum are exact, so the output must match bit for bit.
* The workspace protocol: the arrival counters are zero after every call;
  one workspace serves calls of different split counts in a row; results
  repeat bit for bit; a problem that is not split needs no workspace and
  equals fp8q_gemm."""
import numpy as np
import pytest
import torch

import paper_2609_22870_amd as fp8q
from paper_2609_22870_amd import synth

import _par
import test_gpu_b_gemm as tb
import test_gpu_i_identity as ti

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
PAIRS = tb.PAIRS
# (M, K, N) -> S: 6 tiles of 128 x 128 with 8, 16, 32 K blocks; the last
# tile row ragged (M = 200)
SMALL = {2: (200, 1024, 384), 4: (200, 2048, 384), 8: (200, 4096, 384)}


def splits_of(M, N, K):
    """S from the workspace size (counters padded to 256 bytes, then S
    partial tiles of 64 KB per tile)."""
    ws = fp8q.gemm_splitk_workspace(M, N, K)
    if ws == 0:
        return 1
    tiles = ((M + 127) // 128) * ((N + 127) // 128)
    return (ws - (tiles * 4 + 255) // 256 * 256) // (tiles * 65536)


def test_split_counts():
    for s, (M, K, N) in SMALL.items():
        assert splits_of(M, N, K) == s
    assert splits_of(256, 4096, 12288) == 4
    assert splits_of(256, 12288, 4096) == 1


@pytest.mark.parametrize("splits", list(SMALL))
@pytest.mark.parametrize("pair", list(PAIRS))
def test_splitk_small(pair, splits):
    ga, gb = PAIRS[pair]
    M, K, N = SMALL[splits]
    if gb != fp8q.BLOCK_128x128:
        N += 4                       # ragged last tile column where the pair allows it
    a = synth.activations(M, K, seed=701 + splits, outlier_seed=702, device=DEV)
    b = synth.weights(N, K, seed=703 + splits, device=DEV)
    tb.run_pair(a, b, ga, gb, label="split-K S=%d %s" % (splits, pair), gemm=fp8q.gemm_splitk,
                adds=splits - 1)


def test_splitk_full_8b_decode_down():
    """The 8B FFN down-projection of a decode step: 64 tiles, S = 4, every
    row checked."""
    shape = synth.WORKLOADS["8b_decode_blockwise"]["shapes"][1]
    M, K, N = shape
    assert (M, K, N) == (256, 12288, 4096)
    x = synth.activations(M, K, seed=synth.seed_for(4, 0, 1), outlier_seed=synth.seed_for(4, 3, 1), device=DEV)
    w = synth.weights(N, K, seed=synth.seed_for(4, 1, 1), device=DEV)
    tb.run_pair(x, w, fp8q.BLOCK_1x128, fp8q.BLOCK_128x128, label="split-K decode %s" % (shape,),
                gemm=fp8q.gemm_splitk, adds=3)


ID_SHAPES = {2: (160, 1024, 1024), 4: (200, 2048, 2048), 8: (200, 4096, 1024),
             "decode down": (256, 12288, 4096)}


@pytest.mark.parametrize("shape", list(ID_SHAPES))
@pytest.mark.parametrize("pair", list(PAIRS))
def test_splitk_identity(pair, shape):
    ga, gb = PAIRS[pair]
    M, K, N = ID_SHAPES[shape]
    print("split-K identity pin", pair, shape, (M, K, N), "S =", splits_of(M, N, K), flush=True)
    assert splits_of(M, N, K) > 1
    c = ti.Case(ga, gb, M, K, N, seed=3000 + 11 * list(PAIRS).index(pair) + list(ID_SHAPES).index(shape))
    C = fp8q.gemm_splitk(c.A, c.sA, ga, c.B, c.sB, gb)
    torch.cuda.synchronize()
    ti.check(C.cpu(), c.want(), "split-K %s %s" % (pair, shape))


def _operands(M, K, N, seed):
    a = synth.activations(M, K, seed=seed, outlier_seed=seed + 1, device=DEV)
    b = synth.weights(N, K, seed=seed + 2, device=DEV)
    A, sA = fp8q.quantize(a, fp8q.BLOCK_1x128)
    B, sB = fp8q.quantize(b, fp8q.BLOCK_128x128)
    return A, sA, B, sB


def test_workspace_reuse_and_determinism():
    """One zero-filled workspace, sized for the largest call, serves calls
    with S = 4, 8, 2 and 4 again in a row; every result equals the same call
    on a fresh workspace bit for bit, and the counters (the workspace's
    first bytes) are zero after each call."""
    cases = [(256, 12288, 4096), (200, 4096, 384), (200, 1024, 384), (256, 12288, 4096)]
    need = max(fp8q.gemm_splitk_workspace(M, N, K) for M, K, N in cases)
    ws = torch.zeros(need, dtype=torch.uint8, device=DEV)
    for i, (M, K, N) in enumerate(cases):
        print("workspace reuse", i, (M, K, N), "S =", splits_of(M, N, K), flush=True)
        A, sA, B, sB = _operands(M, K, N, seed=800 + 10 * i)
        got = fp8q.gemm_splitk(A, sA, fp8q.BLOCK_1x128, B, sB, fp8q.BLOCK_128x128, workspace=ws)
        fresh = fp8q.gemm_splitk(A, sA, fp8q.BLOCK_1x128, B, sB, fp8q.BLOCK_128x128)
        torch.cuda.synchronize()
        assert torch.equal(got.view(torch.int16), fresh.view(torch.int16))
        tiles = ((M + 127) // 128) * ((N + 127) // 128)
        assert int(ws[:4 * tiles].count_nonzero()) == 0, "counters not reset"
    # twice on the same inputs and workspace
    A, sA, B, sB = _operands(256, 12288, 4096, seed=900)
    c1 = fp8q.gemm_splitk(A, sA, fp8q.BLOCK_1x128, B, sB, fp8q.BLOCK_128x128, workspace=ws)
    c2 = fp8q.gemm_splitk(A, sA, fp8q.BLOCK_1x128, B, sB, fp8q.BLOCK_128x128, workspace=ws)
    torch.cuda.synchronize()
    assert torch.equal(c1.view(torch.int16), c2.view(torch.int16))


def test_unsplit_problem_is_fp8q_gemm():
    """The 8B decode up-projection has 192 tiles: not split, no workspace,
    the same bits as fp8q_gemm."""
    M, K, N = 256, 4096, 12288
    assert fp8q.gemm_splitk_workspace(M, N, K) == 0
    A, sA, B, sB = _operands(M, K, N, seed=950)
    empty = torch.zeros(16, dtype=torch.uint8, device=DEV)
    got = fp8q.gemm_splitk(A, sA, fp8q.BLOCK_1x128, B, sB, fp8q.BLOCK_128x128, workspace=empty)
    want = fp8q.gemm(A, sA, fp8q.BLOCK_1x128, B, sB, fp8q.BLOCK_128x128)
    torch.cuda.synchronize()
    assert torch.equal(got.view(torch.int16), want.view(torch.int16))


def test_graph_replays_and_side_stream():
    """Captured in a HIP graph (no memset inside: the counters reset
    themselves) and replayed three times, with eager calls of another shape
    through the same workspace, on a stream of their own, in between: every
    replay gives the eager result bit for bit, and the counters are zero
    after each."""
    M, K, N = 256, 12288, 4096
    A, sA, B, sB = _operands(M, K, N, seed=970)
    A2, sA2, B2, sB2 = _operands(200, 4096, 384, seed=980)
    need = max(fp8q.gemm_splitk_workspace(M, N, K), fp8q.gemm_splitk_workspace(200, 384, 4096))
    ws = torch.zeros(need, dtype=torch.uint8, device=DEV)
    eager = fp8q.gemm_splitk(A, sA, fp8q.BLOCK_1x128, B, sB, fp8q.BLOCK_128x128, workspace=ws)
    torch.cuda.synchronize()
    out = torch.empty((M, N), dtype=torch.bfloat16, device=DEV)
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            fp8q.gemm_splitk(A, sA, fp8q.BLOCK_1x128, B, sB, fp8q.BLOCK_128x128, out=out, workspace=ws)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    side = torch.cuda.Stream()
    tiles = ((M + 127) // 128) * ((N + 127) // 128)
    for rep in range(3):
        print("split-K graph replay", rep, flush=True)
        out.fill_(7.0)
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out.view(torch.int16), eager.view(torch.int16)), rep
        assert int(ws[:4 * tiles].count_nonzero()) == 0
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            other = fp8q.gemm_splitk(A2, sA2, fp8q.BLOCK_1x128, B2, sB2, fp8q.BLOCK_128x128, workspace=ws)
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        want = fp8q.gemm_splitk(A2, sA2, fp8q.BLOCK_1x128, B2, sB2, fp8q.BLOCK_128x128)
        torch.cuda.synchronize()
        assert torch.equal(other.view(torch.int16), want.view(torch.int16)), rep


@pytest.mark.parametrize("pair", ["tensor", "row"])
def test_splitk_padded_output(pair):
    """C as the first N columns of a wider buffer (ldc = N + 6, so C rows are
    only 8-byte aligned and the 8-byte store path runs), N not a multiple of
    4: the columns past N stay untouched, the rest match the oracle."""
    ga, gb = PAIRS[pair]
    M, K, N = 200, 2048, 390
    a = synth.activations(M, K, seed=991, outlier_seed=992, device=DEV)
    b = synth.weights(N, K, seed=993, device=DEV)
    assert splits_of(M, N, K) == 4
    tb.run_pair(a, b, ga, gb, label="split-K padded " + pair, pad=6, gemm=fp8q.gemm_splitk, adds=3)
