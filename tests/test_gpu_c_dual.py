"""GPU parity of the dual-layout quantizer (both backward-pass layouts of
Eq. 3, paper Sec. 2.2, from one read) against the oracle: its outputs must be
the oracle's 1x128 quantization and its transposed 128x1 quantization, bit
for bit.  Calls go through the C-ABI."""
import numpy as np
import pytest
import torch

import paper_2609_22870_amd as fp8q
from paper_2609_22870_amd import synth

import _par

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def oracle_pair(x):
    bits = synth.bf16_bits(x)
    cr, sr = _par.quantize(bits, fp8q.BLOCK_1x128)
    ct, st = _par.quantize(bits, fp8q.BLOCK_128x1, transposed=True)
    return cr, sr, ct, st


def assert_same_bits(got, want, what):
    got = np.asarray(got)
    assert got.shape == want.shape, (what, got.shape, want.shape)
    if got.dtype == np.float32:
        got, want = got.view(np.uint32), want.view(np.uint32)
    bad = np.argwhere(got != want)
    assert bad.size == 0, "%s differ at %s" % (what, bad[:5].tolist())


def check(x, label):
    print("dual quantize parity", label, tuple(x.shape), flush=True)
    out = fp8q.quantize_dual(x.to(DEV))
    torch.cuda.synchronize()
    want = oracle_pair(x)
    for g, w, name in zip(out, want, ("row codes", "row scales", "transposed codes", "transposed scales")):
        assert_same_bits(g.cpu().numpy(), w, name)


def test_small_several_tiles():
    check(synth.activations(384, 512, seed=41, outlier_seed=42), "activations")
    check(synth.grads(256, 640, seed=43), "gradients")


def test_special_units():
    """Units that take the other branches of the cast: an all-zero row block
    and column block (S = 1), a column whose amax is an fp32 subnormal (the
    IEEE-division path), and single non-zero units (code 448)."""
    x = synth.activations(256, 384, seed=45, outlier_seed=46)
    x[3, 128:256] = 0.0                        # zero 1x128 unit
    x[128:256, 7] = 0.0                        # zero 128x1 unit
    x[:128, 200] = torch.tensor(2.0 ** -130).to(torch.bfloat16)  # subnormal amax
    x[5, :128] = 0.0
    x[5, 17] = -3.5                            # single non-zero row unit
    check(x, "special units")


def test_matches_single_layout_kernels():
    """Same bytes as the two single-layout calls of fp8q_quantize."""
    x = synth.grads(512, 1024, seed=47).to(DEV)
    cr, sr, ct, st = fp8q.quantize_dual(x)
    r = fp8q.quantize(x, fp8q.BLOCK_1x128)
    t = fp8q.quantize(x, fp8q.BLOCK_128x1, transposed=True)
    torch.cuda.synchronize()
    assert torch.equal(cr, r[0]) and torch.equal(sr.view(torch.int32), r[1].view(torch.int32))
    assert torch.equal(ct, t[0]) and torch.equal(st.view(torch.int32), t[1].view(torch.int32))


def test_padded_leading_dimensions():
    x = synth.activations(256, 256, seed=49, outlier_seed=50)
    xd = torch.zeros((256, 320), dtype=torch.bfloat16, device=DEV)
    xd[:, :256] = x.to(DEV)
    codes_r = torch.full((256, 272), 0x5A, dtype=torch.uint8, device=DEV)
    codes_t = torch.full((256, 288), 0x5A, dtype=torch.uint8, device=DEV)
    sr = torch.empty(fp8q.scales_count(256, 256, fp8q.BLOCK_1x128), dtype=torch.float32, device=DEV)
    st = torch.empty(fp8q.scales_count(256, 256, fp8q.BLOCK_128x1, True), dtype=torch.float32, device=DEV)
    fp8q.quantize_dual(xd[:, :256], codes_r[:, :256], sr, codes_t[:, :256], st)
    torch.cuda.synchronize()
    want = oracle_pair(x)
    assert_same_bits(codes_r[:, :256].cpu().numpy(), want[0], "row codes")
    assert_same_bits(sr.cpu().numpy(), want[1], "row scales")
    assert_same_bits(codes_t[:, :256].cpu().numpy(), want[2], "transposed codes")
    assert_same_bits(st.cpu().numpy(), want[3], "transposed scales")
    assert torch.all(codes_r[:, 256:] == 0x5A) and torch.all(codes_t[:, 256:] == 0x5A)


def test_deterministic():
    x = synth.grads(256, 512, seed=51).to(DEV)
    a = fp8q.quantize_dual(x)
    b = fp8q.quantize_dual(x)
    torch.cuda.synchronize()
    for u, v in zip(a, b):
        assert torch.equal(u.view(torch.uint8), v.view(torch.uint8))


@pytest.mark.parametrize("name,rows,cols", [("32B dY 16384x25600", 16384, 25600),
                                            ("8B X 16384x4096", 16384, 4096)])
def test_full_size(name, rows, cols):
    """The backward-pass operands at full size: the 32B FFN output gradient
    and the 8B FFN input, every byte against the oracle."""
    if "dY" in name:
        x = synth.grads(rows, cols, seed=synth.seed_for(5, 2))
    else:
        x = synth.activations(rows, cols, seed=synth.seed_for(2, 0), outlier_seed=synth.seed_for(2, 3))
    check(x, name)
