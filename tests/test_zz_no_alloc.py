"""The allocation-free entry point fp8q_calibrate_clip_noalloc against the
workspace entry point fp8q_calibrate_clip, through the C-ABI: two calls in a
row on one device, the second on a smaller batch (fewer blocks of partial
sums, so it reads a layout the first call's stale partials do not match),
on the null stream and on a stream of its own.  Both entry points run the
same kernels over partials in the same layout, so every field of the
result is bitwise equal; the first batch is also held to the oracle
(Sec. 4, Alg. 1, Eq. 5) as the workspace entry point's parity tests do."""
import numpy as np
import pytest
import torch

import paper_2609_22870_amd as fp8q
from paper_2609_22870_amd import synth
from oracle import clip

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
KEYS = ("adv", "w_tis", "pi_sampler", "r_bf16", "r_fp8")


def _both(b, l_old, h_old, stream=None):
    ts = [b[k].to(DEV) for k in KEYS]
    res_ws = torch.full((80,), 0x5A, dtype=torch.uint8, device=DEV)
    res_na = torch.full((80,), 0xA5, dtype=torch.uint8, device=DEV)
    torch.cuda.synchronize()
    ctx = torch.cuda.stream(stream) if stream is not None else torch.cuda.stream(torch.cuda.current_stream())
    with ctx:
        fp8q.calibrate_clip(*ts, l_old, h_old, result=res_ws, read=False)
        fp8q.calibrate_clip_noalloc(*ts, l_old, h_old, result=res_na, read=False)
    torch.cuda.synchronize()
    return res_ws, res_na


def _fields(buf):
    raw = buf.cpu().numpy().tobytes()
    f = np.frombuffer(raw[:56], dtype=np.float64)
    return dict(zip(("l_new", "h_new", "l_star", "h_star", "alpha_low", "rho_bf16", "rho_fp8"), f.tolist()))


@pytest.mark.parametrize("on_stream", [False, True])
def test_noalloc_matches_workspace_entry(on_stream):
    big = synth.rl_batch(64, 8, seed=91, fp8_sigma=0.1)
    small = synth.rl_batch(4, 8, seed=92, fp8_sigma=0.1, min_len=1, max_len=3000)
    assert small["adv"].numel() < big["adv"].numel()
    stream = torch.cuda.Stream() if on_stream else None
    for i, (b, lo, hi) in enumerate(((big, 0.6, 1.8), (small, 0.66, 1.5))):
        n = b["adv"].numel()
        print("noalloc clip call", i, n, "tokens", "stream" if on_stream else "null stream", flush=True)
        res_ws, res_na = _both(b, lo, hi, stream)
        assert torch.equal(res_ws, res_na), (_fields(res_ws), _fields(res_na))
        if i == 0:
            want = clip.calibrate(*(b[k].numpy() for k in KEYS), lo, hi, clip.PAPER_CONFIG)
            got = _fields(res_na)
            assert got["l_new"] == want["l_new"] and got["h_new"] == want["h_new"]
            assert got["l_star"] == want["l_star"] and got["h_star"] == want["h_star"]


def test_noalloc_rejects_before_launch():
    b = {k: v.to(DEV) for k, v in synth.rl_batch(2, 8, seed=93).items()}
    with pytest.raises(fp8q.Fp8qError):
        fp8q.calibrate_clip_noalloc(*(b[k] for k in KEYS), 0.6, 1.8,
                                    config=dict(fp8q.PAPER_CLIP_CONFIG, l_min=0.42))
