"""GPU parity of the grouped GEMM (several FP8 linear-layer products in one
launch: the fused query / key / value and gate / up projections) through
the C-ABI.  Each problem's output must equal fp8q_gemm's for the same
operands bit for bit (the per-element arithmetic does not depend on the
tile), and the oracle's exact product to the GEMM tolerance."""
import numpy as np
import pytest
import torch

import paper_2609_22870_amd as fp8q
from paper_2609_22870_amd import synth

import _par

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
TOL = 4e-3


def check_group(a_list, w_list, ga, gb, rows=None, label=""):
    """Quantize every activation and weight, run the problems (a_i, w_i)
    grouped and one by one, and compare."""
    print("grouped gemm", label, [tuple(a.shape) for a in a_list], [tuple(w.shape) for w in w_list], flush=True)
    qa = {}
    probs = []
    for a, w in zip(a_list, w_list):
        if id(a) not in qa:
            qa[id(a)] = fp8q.quantize(a, ga)
        A, sA = qa[id(a)]
        B, sB = fp8q.quantize(w, gb)
        probs.append((A, sA, B, sB))
    outs = fp8q.gemm_grouped(probs, ga, gb)
    singles = [fp8q.gemm(A, sA, ga, B, sB, gb) for A, sA, B, sB in probs]
    torch.cuda.synchronize()
    for i, (c, c1) in enumerate(zip(outs, singles)):
        assert torch.equal(c.view(torch.int16), c1.view(torch.int16)), "problem %d differs from fp8q_gemm" % i
    for i, (a, w, c) in enumerate(zip(a_list, w_list, outs)):
        r = np.arange(a.shape[0]) if rows is None else rows
        idx = torch.as_tensor(r, device=a.device)
        src = a if ga == fp8q.TENSOR else a[idx]
        oA, osA = _par.quantize(synth.bf16_bits(src.cpu()), ga)
        oB, osB = _par.quantize(synth.bf16_bits(w.cpu()), gb)
        ref = _par.gemm_rows(oA, osA, ga, oB, osB, gb, r if ga == fp8q.TENSOR else np.arange(len(r)))
        kind = "accumulate" if ga in (fp8q.TENSOR, fp8q.ROW) else "promote"
        _par.check_gemm(c.float().cpu().numpy()[r], ref, oA[r] if ga == fp8q.TENSOR else oA, osA, ga,
                        oB, osB, gb, kind, tol=TOL, label="problem %d" % i)


@pytest.mark.parametrize("ga,gb", [(fp8q.BLOCK_1x128, fp8q.BLOCK_128x128), (fp8q.ROW, fp8q.ROW),
                                   (fp8q.TENSOR, fp8q.TENSOR)])
def test_qkv_shared_input_small(ga, gb):
    """Query, key and value projections (4 : 1 : 1 widths) of one input with
    a ragged token count."""
    x = synth.activations(1000, 512, seed=201, outlier_seed=202, device=DEV)
    ws = [synth.weights(n, 512, seed=203 + i, device=DEV) for i, n in enumerate((512, 128, 128))]
    check_group([x, x, x], ws, ga, gb, label="qkv small")


def test_mixed_tiled_and_k_group_problems():
    """A large problem (128 x 128 or larger tiles) and a skinny one that a
    single call splits into two K groups: the grouped call runs them in two
    launches, each output still fp8q_gemm's bit for bit."""
    x1 = synth.activations(4096, 512, seed=211, outlier_seed=212, device=DEV)
    x2 = synth.activations(192, 512, seed=213, outlier_seed=214, device=DEV)
    w1 = synth.weights(2048, 512, seed=215, device=DEV)
    w2 = synth.weights(384, 512, seed=216, device=DEV)
    check_group([x1, x2], [w1, w2], fp8q.BLOCK_1x128, fp8q.BLOCK_128x128, rows=_par.sample_rows(192),
                label="mixed tiled and K groups")


def test_distinct_inputs_and_sizes():
    """Problems with their own inputs, token counts and widths (every tile
    size of one launch is the same; the problems' rasters follow each other)."""
    xs = [synth.activations(m, 384, seed=211 + i, outlier_seed=221 + i, device=DEV)
          for i, m in enumerate((130, 700, 64, 1500))]
    ws = [synth.weights(n, 384, seed=231 + i, device=DEV) for i, n in enumerate((256, 384, 128, 640))]
    check_group(xs, ws, fp8q.BLOCK_1x128, fp8q.BLOCK_128x128, label="distinct")


def test_eight_problems_128_tiles():
    """FP8Q_MAX_GROUP problems, enough tiles for the 128 x 128 tile."""
    x = synth.activations(2048, 256, seed=241, outlier_seed=242, device=DEV)
    ws = [synth.weights(512, 256, seed=243 + i, device=DEV) for i in range(fp8q.MAX_GROUP)]
    check_group([x] * fp8q.MAX_GROUP, ws, fp8q.BLOCK_1x128, fp8q.BLOCK_128x128,
                rows=_par.sample_rows(2048), label="eight")


def test_too_many_problems_refused():
    a = torch.zeros((128, 128), dtype=torch.uint8, device=DEV)
    s = torch.ones(128, dtype=torch.float32, device=DEV)
    with pytest.raises(ValueError):
        fp8q.gemm_grouped([(a, s, a, s)] * (fp8q.MAX_GROUP + 1), fp8q.ROW, fp8q.ROW)


@pytest.mark.parametrize("kind", ["qkv", "gate_up"])
def test_full_8b_fused_projections(kind):
    """The 8B-class model's fused projections over 16384 tokens: query, key
    and value (4096, 1024, 1024 outputs) or gate and up (12288 each), from
    X 16384 x 4096, blockwise."""
    x = synth.activations(16384, 4096, seed=synth.seed_for(6, 0), outlier_seed=synth.seed_for(6, 3), device=DEV)
    widths = (4096, 1024, 1024) if kind == "qkv" else (12288, 12288)
    ws = [synth.weights(n, 4096, seed=synth.seed_for(6, 1, i), device=DEV) for i, n in enumerate(widths)]
    check_group([x] * len(ws), ws, fp8q.BLOCK_1x128, fp8q.BLOCK_128x128,
                rows=_par.sample_rows(16384, per_band=1), label="8B " + kind)
