"""Pins of the Calibrated Clipping oracle (paper Sec. 4, Alg. 1, Eq. 5)
against things fixed independently of its code: an exact rational
brute force on small batches, closed forms of SmoothUpdate, cases whose
answer follows from the definitions (identical ratios, uniformly scaled
ratios), invariances, and the degenerate batches."""
from fractions import Fraction

import numpy as np
import pytest

from oracle import clip

CFG = clip.PAPER_CONFIG


def batch(n, seed, zero_frac=0.1, fp8_sigma=0.03):
    rng = np.random.default_rng(seed)
    a = rng.standard_normal(n).astype(np.float32)
    a[rng.random(n) < zero_frac] = 0.0
    w = np.minimum(np.exp(0.02 * rng.standard_normal(n)), 2.0).astype(np.float32)
    pi = (1.0 / (1.0 + np.exp(-(3.0 + 2.0 * rng.standard_normal(n))))).astype(np.float32)
    rb = np.exp(0.1 * rng.standard_normal(n)).astype(np.float32)
    rf = (rb * np.exp(fp8_sigma * rng.standard_normal(n))).astype(np.float32)
    return a, w, pi, rb, rf


def brute_force(a, w, pi, rb, rf, l_old, h_old, cfg):
    """Alg. 1 with exact rational sums and explicit loops (first minimum on
    ties).  Grid points are the float64 numbers lo + k * step."""
    F = Fraction
    lg = [cfg["l_min"] + k * cfg["step"] for k in range(int(round((cfg["l_max"] - cfg["l_min"]) / cfg["step"])) + 1)]
    hg = [cfg["h_min"] + k * cfg["step"] for k in range(int(round((cfg["h_max"] - cfg["h_min"]) / cfg["step"])) + 1)]
    toks = [(F(float(a[i])), F(float(w[i])), F(float(pi[i])), F(float(rb[i])), F(float(rf[i]))) for i in range(len(a))]
    neg = [t for t in toks if t[0] < 0]
    if not neg:
        return None

    def ratio(r_index, lo, hi):
        num = sum((t[1] * t[2] * t[r_index] * t[0] for t in toks if t[0] > 0 and t[r_index] < F(hi)), F(0))
        den = sum((t[1] * t[2] * t[r_index] * t[0] for t in toks if t[0] < 0 and t[r_index] > F(lo)), F(0))
        return None if den == 0 else abs(num) / abs(den)

    cnt_ref = sum(1 for t in neg if t[3] <= F(cfg["c_low_ref"]))
    best = None
    for k, L in enumerate(lg):
        d = abs(sum(1 for t in neg if t[4] <= F(L)) - cnt_ref)
        if best is None or d < best[0]:
            best = (d, k)
    l_star = lg[best[1]]
    rho_ref = ratio(3, cfg["c_low_ref"], cfg["c_high_ref"])
    h_star = None
    if rho_ref is not None:
        best = None
        for k, H in enumerate(hg):
            v = ratio(4, l_star, H)
            if v is None:
                break
            d = abs(v - rho_ref)
            if best is None or d < best[0]:
                best = (d, k)
        if best is not None:
            h_star = hg[best[1]]
    return dict(l_star=l_star, h_star=h_star, alpha_low=F(cnt_ref, len(neg)), rho_bf16=rho_ref)


@pytest.mark.parametrize("seed", range(6))
def test_matches_exact_brute_force(seed):
    a, w, pi, rb, rf = batch(300, seed)
    got = clip.calibrate(a, w, pi, rb, rf, 0.6, 1.8)
    want = brute_force(a, w, pi, rb, rf, 0.6, 1.8, CFG)
    assert got["l_star"] == want["l_star"]
    assert got["h_star"] == want["h_star"]
    assert got["alpha_low"] == float(want["alpha_low"])
    assert abs(got["rho_bf16"] - float(want["rho_bf16"])) <= 1e-13 * float(want["rho_bf16"])
    assert got["l_new"] == clip.smooth_update(0.6, want["l_star"], CFG["delta_l"])


def test_smooth_update_closed_forms():
    # b + clip((b* - b) / 2, -delta, delta)
    assert clip.smooth_update(0.6, 0.8, 0.05) == 0.65           # capped at +delta
    assert clip.smooth_update(0.6, 0.64, 0.05) == 0.6 + 0.02    # half the distance
    assert clip.smooth_update(1.8, 1.24, 0.1) == 1.7            # capped at -delta
    assert clip.smooth_update(1.3, 1.3, 0.1) == 1.3             # at the target
    assert clip.smooth_update(0.7, 0.66, 0.05) == 0.7 - 0.02


def test_grids_of_the_paper():
    lg, hg = clip.grid(0.5, 0.9, 0.02), clip.grid(1.2, 2.0, 0.02)
    assert len(lg) == 21 and len(hg) == 41
    assert lg[0] == 0.5 and lg[-1] == 0.9 and lg[15] == 0.8
    assert hg[0] == 1.2 and hg[-1] == 2.0 and hg[2] == 1.24


def test_identical_ratios_recover_the_reference_bounds():
    """With r_FP8 = r_BF16 the FP8 CDF is the BF16 one, so L* is the grid
    point c_low_ref = 0.8, and at L* = 0.8 the FP8 ratio of Eq. 5 at H = 1.24
    is the reference ratio itself: H* = 1.24.  The smoothed bounds then move
    from the paper's start [0.6, 1.8] by at most delta_L, delta_H."""
    a, w, pi, rb, _ = batch(20000, 7)
    got = clip.calibrate(a, w, pi, rb, rb, 0.6, 1.8)
    assert got["l_star"] == 0.8 and got["h_star"] == 1.24
    assert got["rho_fp8"] == got["rho_bf16"]
    assert got["l_new"] == 0.65 and got["h_new"] == 1.7


def test_uniformly_lower_fp8_ratios_lower_the_bound():
    """r_FP8 = 0.9 r_BF16 (exact in float32 for these draws is not needed:
    F_FP8(L) = F_BF16(L / 0.9) up to rounding), so L* is the grid point
    nearest 0.8 * 0.9 = 0.72."""
    a, w, pi, rb, _ = batch(50000, 8)
    rf = (rb.astype(np.float64) * 0.9).astype(np.float32)
    got = clip.calibrate(a, w, pi, rb, rf, 0.6, 1.8)
    assert got["l_star"] == clip.grid(0.5, 0.9, 0.02)[11]       # 0.72


def test_noisier_fp8_ratios_relax_the_lower_bound():
    """The failure the paper describes: FP8 noise widens the ratio spread,
    so more negative tokens fall below 0.8 than under BF16; matching the
    quantile moves L* below 0.8."""
    a, w, pi, rb, rf = batch(50000, 9, fp8_sigma=0.1)
    got = clip.calibrate(a, w, pi, rb, rf, 0.6, 1.8)
    assert got["l_star"] < 0.8


def test_zero_advantage_tokens_change_nothing():
    a, w, pi, rb, rf = batch(3000, 10, zero_frac=0.0)
    base = clip.calibrate(a, w, pi, rb, rf, 0.6, 1.8)
    rng = np.random.default_rng(11)
    extra = 500
    a2 = np.concatenate([a, np.zeros(extra, np.float32)])
    w2 = np.concatenate([w, rng.random(extra).astype(np.float32)])
    pi2 = np.concatenate([pi, rng.random(extra).astype(np.float32)])
    rb2 = np.concatenate([rb, (0.3 + 2 * rng.random(extra)).astype(np.float32)])
    rf2 = np.concatenate([rf, (0.3 + 2 * rng.random(extra)).astype(np.float32)])
    got = clip.calibrate(a2, w2, pi2, rb2, rf2, 0.6, 1.8)
    for key in ("l_star", "h_star", "alpha_low", "n_neg", "n_pos"):
        assert got[key] == base[key], key
    assert got["rho_bf16"] == base["rho_bf16"]


def test_positive_scaling_of_advantages():
    """Counts do not see the advantage's size and Eq. 5 is a ratio, so
    scaling every A by 4 (exact) keeps L* and H* and rho."""
    a, w, pi, rb, rf = batch(4000, 12)
    base = clip.calibrate(a, w, pi, rb, rf, 0.6, 1.8)
    got = clip.calibrate(a * np.float32(4.0), w, pi, rb, rf, 0.6, 1.8)
    assert got["l_star"] == base["l_star"] and got["h_star"] == base["h_star"]
    assert got["rho_bf16"] == base["rho_bf16"]


def test_degenerate_batches_keep_the_bounds():
    a, w, pi, rb, rf = batch(1000, 13)
    pos_only = np.abs(a)
    got = clip.calibrate(pos_only, w, pi, rb, rf, 0.62, 1.74)
    assert (got["l_new"], got["h_new"]) == (0.62, 1.74)
    assert not got["l_updated"] and not got["h_updated"]
    # only negative tokens, every ratio far below 0.8: L still moves (the
    # counts are defined), but no token has r > c_low_ref, so the BF16
    # denominator of Eq. 5 is zero, rho is undefined and H keeps its value
    neg_low = -np.abs(a)
    got = clip.calibrate(neg_low, w, pi, rb * np.float32(0.1), rf * np.float32(0.1), 0.62, 1.74)
    assert got["l_updated"] and not got["h_updated"] and got["h_new"] == 1.74
