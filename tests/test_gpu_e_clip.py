"""GPU parity of Calibrated Clipping (paper Sec. 4, Alg. 1, Eq. 5) against
the float64 oracle, through the C-ABI.

Both sides take the same decisions: the lower-bound search compares integer
counts (exact on both sides), and the upper-bound search compares float64
ratios whose sums differ only in summation order (the GPU sums in a fixed
tree), so the grid optima, the counts and the new bounds must be equal and
the Eq. 5 ratios equal to 1e-12 relative."""
import math

import numpy as np
import pytest
import torch

import paper_2609_22870_amd as fp8q
from paper_2609_22870_amd import synth
from oracle import clip

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
KEYS = ("adv", "w_tis", "pi_sampler", "r_bf16", "r_fp8")


def compare(b, l_old, h_old, config=None, label=""):
    n = b["adv"].numel()
    print("calibrated clipping parity", label, n, "tokens", flush=True)
    cfg = config or clip.PAPER_CONFIG
    got = fp8q.calibrate_clip(*(b[k].to(DEV) for k in KEYS), l_old, h_old, config=cfg)
    want = clip.calibrate(*(b[k].numpy() for k in KEYS), l_old, h_old, cfg)
    print("  L* %r H* %r -> [%r, %r]" % (got["l_star"], got["h_star"], got["l_new"], got["h_new"]), flush=True)
    assert got["n_neg"] == want["n_neg"] and got["n_pos"] == want["n_pos"]
    assert bool(got["l_updated"]) == want["l_updated"] and bool(got["h_updated"]) == want["h_updated"]
    for k in ("l_star", "h_star", "alpha_low"):
        if want[k] is None:
            assert math.isnan(got[k]), k
        else:
            assert got[k] == want[k], (k, got[k], want[k])
    for k in ("rho_bf16", "rho_fp8"):
        if want[k] is None:
            assert math.isnan(got[k]), k
        else:
            assert abs(got[k] - want[k]) <= 1e-12 * abs(want[k]), (k, got[k], want[k])
    assert got["l_new"] == want["l_new"] and got["h_new"] == want["h_new"]
    return got


def test_paper_batch():
    """One batch of the paper's GRPO setup (256 prompts x 8 responses,
    8.9 M tokens), bounds from the paper's initialisation."""
    b = synth.rl_batch(**synth.RL_BATCH, seed=5001)
    compare(b, 0.6, 1.8, label="paper batch")


@pytest.mark.parametrize("prompts,ratio_sigma,fp8_sigma,seed", [(256, 0.12, 0.06, 5101), (64, 0.2, 0.1, 5102),
                                                                 (64, 0.12, 0.03, 5103)])
def test_lower_search_in_the_body(prompts, ratio_sigma, fp8_sigma, seed):
    """BF16 ratios spread widely enough that a few percent or more of the
    negative-advantage tokens sit at or below c_low_ref = 0.8 (the BF16
    importance ratios of off-policy batches), so that stage 1 of Alg. 1
    matches counts in the body of the distribution, not in its far tail,
    and L* lands inside the grid; the first batch is of the paper's size."""
    b = synth.rl_batch(prompts, 8, seed=seed, ratio_sigma=ratio_sigma, fp8_sigma=fp8_sigma)
    got = compare(b, 0.6, 1.8, label="ratio sigma %g, fp8 sigma %g" % (ratio_sigma, fp8_sigma))
    print("  alpha_low %.4f" % got["alpha_low"], flush=True)
    assert 0.01 <= got["alpha_low"] <= 0.2
    assert 0.5 < got["l_star"] < 0.9


@pytest.mark.parametrize("seed,fp8_sigma,l_old,h_old", [(11, 0.03, 0.66, 1.5), (12, 0.1, 0.72, 1.3),
                                                        (13, 0.2, 0.55, 1.95)])
def test_smaller_batches(seed, fp8_sigma, l_old, h_old):
    b = synth.rl_batch(32, 8, seed=seed, fp8_sigma=fp8_sigma)
    compare(b, l_old, h_old, label="seed %d sigma %g" % (seed, fp8_sigma))


@pytest.mark.parametrize("n", [1, 3, 1021, 4096 + 5, 3 * 5120 + 1])
def test_ragged_lengths(n):
    """Token counts that leave a partial 4-token group, a partial block, or
    a single token."""
    b = synth.rl_batch(4, 8, seed=21 + n, min_len=1, max_len=4000)
    b = {k: v[:n].clone() for k, v in b.items()}
    if b["adv"].numel() < n:
        pytest.skip("batch shorter than %d" % n)
    compare(b, 0.6, 1.8, label="n=%d" % n)


def test_identical_ratios():
    b = synth.rl_batch(16, 8, seed=31)
    b["r_fp8"] = b["r_bf16"].clone()
    got = compare(b, 0.6, 1.8, label="identical ratios")
    assert got["l_star"] == 0.8 and got["h_star"] == 1.24


def test_degenerate_batches():
    b = synth.rl_batch(8, 8, seed=41)
    b["adv"] = b["adv"].abs()                      # no negative advantage
    got = compare(b, 0.62, 1.74, label="no negatives")
    assert not got["l_updated"] and got["l_new"] == 0.62 and got["h_new"] == 1.74
    b = synth.rl_batch(8, 8, seed=42)
    b["adv"] = -b["adv"].abs() - 1e-3             # no positive advantage: rho = 0
    compare(b, 0.62, 1.74, label="no positives")


def test_general_grid():
    """A grid beyond the paper's sizes (24 lower, 48 upper points) runs the
    general instantiation; one more point is refused."""
    cfg = dict(clip.PAPER_CONFIG, l_min=0.44, l_max=0.9, h_min=1.1, h_max=2.04)
    b = synth.rl_batch(32, 8, seed=51, fp8_sigma=0.1)
    compare(b, 0.6, 1.8, config=cfg, label="24 x 48 grid")
    with pytest.raises(fp8q.Fp8qError):
        fp8q.calibrate_clip(*(b[k].to(DEV) for k in KEYS), 0.6, 1.8,
                            config=dict(cfg, l_min=0.42))


def test_deterministic():
    b = {k: v.to(DEV) for k, v in synth.rl_batch(64, 8, seed=61).items()}
    res = [torch.empty(80, dtype=torch.uint8, device=DEV) for _ in range(2)]
    for r in res:
        fp8q.calibrate_clip(*(b[k] for k in KEYS), 0.6, 1.8, result=r)
    torch.cuda.synchronize()
    assert torch.equal(res[0], res[1])


def _result_dict(buf):
    """The fp8q_clip_result fields of an 80-byte device buffer."""
    raw = buf.cpu().numpy().tobytes()
    f = np.frombuffer(raw[:56], dtype=np.float64)
    i = np.frombuffer(raw[56:72], dtype=np.int64)
    u = np.frombuffer(raw[72:80], dtype=np.int32)
    return dict(zip(("l_new", "h_new", "l_star", "h_star", "alpha_low", "rho_bf16", "rho_fp8"), f.tolist()),
                n_neg=int(i[0]), n_pos=int(i[1]), l_updated=int(u[0]), h_updated=int(u[1]))


def test_stale_and_reused_workspace():
    """A workspace full of stale bytes, then reused for a batch of another
    size (another block count) and again: the oracle's answer each time."""
    big = synth.rl_batch(64, 8, seed=71, fp8_sigma=0.1)
    small = synth.rl_batch(8, 8, seed=72, fp8_sigma=0.1)
    need = fp8q.lib().fp8q_calibrate_clip_workspace(big["adv"].numel())
    ws = torch.full((need,), 0xFF, dtype=torch.uint8, device=DEV)
    for b, label in ((big, "stale workspace"), (small, "reused workspace"), (big, "reused again")):
        print("calibrated clipping", label, b["adv"].numel(), "tokens", flush=True)
        res = torch.empty(80, dtype=torch.uint8, device=DEV)
        fp8q.calibrate_clip(*(b[k].to(DEV) for k in KEYS), 0.6, 1.8, workspace=ws, result=res, read=False)
        torch.cuda.synchronize()
        got = _result_dict(res)
        want = clip.calibrate(*(b[k].numpy() for k in KEYS), 0.6, 1.8, clip.PAPER_CONFIG)
        assert got["n_neg"] == want["n_neg"] and got["n_pos"] == want["n_pos"]
        assert got["l_new"] == want["l_new"] and got["h_new"] == want["h_new"]
        assert got["l_star"] == want["l_star"] and got["h_star"] == want["h_star"]


def test_graph_replays():
    """Captured in a HIP graph and replayed three times, with eager calls on
    other data through the same workspace in between: every replay gives
    the eager result."""
    b = {k: v.to(DEV) for k, v in synth.rl_batch(32, 8, seed=81, fp8_sigma=0.1).items()}
    other = {k: v.to(DEV) for k, v in synth.rl_batch(16, 8, seed=82).items()}
    need = fp8q.lib().fp8q_calibrate_clip_workspace(b["adv"].numel())
    ws = torch.empty(need, dtype=torch.uint8, device=DEV)
    eager = torch.empty(80, dtype=torch.uint8, device=DEV)
    fp8q.calibrate_clip(*(b[k] for k in KEYS), 0.6, 1.8, workspace=ws, result=eager, read=False)
    torch.cuda.synchronize()
    res = torch.full((80,), 0x5A, dtype=torch.uint8, device=DEV)
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            fp8q.calibrate_clip(*(b[k] for k in KEYS), 0.6, 1.8, workspace=ws, result=res, read=False)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    scratch = torch.empty(80, dtype=torch.uint8, device=DEV)
    for rep in range(3):
        print("graph replay", rep, flush=True)
        res.fill_(0x5A)
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(res, eager), rep
        fp8q.calibrate_clip(*(other[k] for k in KEYS), 0.6, 1.8, workspace=ws, result=scratch, read=False)
        torch.cuda.synchronize()
