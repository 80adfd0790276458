"""Oracle for Calibrated Clipping (paper Sec. 4, Alg. 1, Eq. 5).

TEST INFRASTRUCTURE ONLY, like the rest of ``oracle/``: plain numpy in
float64, written from the method's definitions in the order the paper states
its steps.  Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline
leg of ``bench.py`` may use it; it shares no code with the HIP library.

Inputs are per-token float32 arrays of one training batch: advantages A,
TIS weights w (already truncated at C), the sampler's token probabilities
pi_sampler, and the importance ratios under the BF16 and the FP8 forward
passes.  Readings of points the paper leaves open (each also listed in the
design notes):

* The CDF is F(x) = (number of negative-advantage tokens with r <= x) /
  (number of negative-advantage tokens): "<=", the usual CDF.
* Tokens with A = 0 belong to neither sum of Eq. 5 nor to the negative CDF.
* The search grid of an interval [lo, hi] with step d is lo + k * d for
  k = 0 .. round((hi - lo) / d), each point rounded to float64 once after
  the product and once after the sum (no fused multiply-add).
* Ties in either search go to the first (smallest) grid point.
* Eq. 5 weights each token by pi_sampler (as printed in Eq. 5), and each
  term is the float64 product ((w * pi) * r) * A.
* The lower-bound search matches counts: minimising |F_FP8(L) - alpha_low|
  over the grid is minimising |#{r_FP8 <= L} - #{r_BF16 <= c_low_ref}| over
  the negative-advantage tokens, an exact integer comparison.
* Degenerate batches: with no negative-advantage token F is undefined and
  both bounds keep their old values; when a denominator of Eq. 5 is zero
  (for the BF16 reference, or for the FP8 ratio at L*), rho is undefined
  and the upper bound keeps its old value.
"""
import numpy as np

# The paper's settings (Sec. 4): search intervals, step, update limits; the
# GRPO experiments' reference bounds (Sec. 5.1).
PAPER_CONFIG = dict(c_low_ref=0.8, c_high_ref=1.24, l_min=0.5, l_max=0.9, h_min=1.2, h_max=2.0,
                    step=0.02, delta_l=0.05, delta_h=0.1)
PAPER_INIT = (0.6, 1.8)


def grid(lo, hi, step):
    """Search grid points lo + k * step, k = 0 .. round((hi - lo) / step)."""
    n = int(round((hi - lo) / step)) + 1
    k = np.arange(n, dtype=np.float64)
    return (k * np.float64(step)) + np.float64(lo)


def smooth_update(b, b_star, delta):
    """SmoothUpdate(b, b*, delta) = b + clip((b* - b) / 2, -delta, delta)."""
    step = (np.float64(b_star) - np.float64(b)) / 2.0
    return float(np.float64(b) + min(max(step, -np.float64(delta)), np.float64(delta)))


def update_terms(a, w, pi, r):
    """Per-token terms w * pi * r * A of Eq. 5, in float64."""
    a, w, pi, r = (np.asarray(v, dtype=np.float32).astype(np.float64) for v in (a, w, pi, r))
    return ((w * pi) * r) * a


def rho(a, w, pi, r, c_low, c_high):
    """Eq. 5: |sum over A>0 of w pi r A [r < c_high]| / |sum over A<0 of
    w pi r A [r > c_low]|; also returns numerator and denominator."""
    a = np.asarray(a, dtype=np.float32)
    r64 = np.asarray(r, dtype=np.float32).astype(np.float64)
    t = update_terms(a, w, pi, r)
    num = abs(float(np.sum(t[(a > 0) & (r64 < c_high)])))
    den = abs(float(np.sum(t[(a < 0) & (r64 > c_low)])))
    return (num / den if den > 0 else None), num, den


def calibrate(a, w, pi, r_bf16, r_fp8, l_old, h_old, cfg=PAPER_CONFIG):
    """Alg. 1: the new clipping bounds (L_new, H_new) and the statistics the
    steps produce, as a dict."""
    a = np.asarray(a, dtype=np.float32)
    rb = np.asarray(r_bf16, dtype=np.float32).astype(np.float64)
    rf = np.asarray(r_fp8, dtype=np.float32).astype(np.float64)
    neg, pos = a < 0, a > 0
    n_neg, n_pos = int(neg.sum()), int(pos.sum())
    out = dict(n_neg=n_neg, n_pos=n_pos, l_new=float(l_old), h_new=float(h_old), l_star=None,
               h_star=None, alpha_low=None, rho_bf16=None, rho_fp8=None, l_updated=False,
               h_updated=False)
    if n_neg == 0:
        return out

    # high-precision reference statistics
    cnt_ref = int(np.sum(rb[neg] <= cfg["c_low_ref"]))
    out["alpha_low"] = cnt_ref / n_neg
    rho_ref, _, _ = rho(a, w, pi, r_bf16, cfg["c_low_ref"], cfg["c_high_ref"])
    out["rho_bf16"] = rho_ref

    # lower bound: match the clipped quantile of the negative tokens
    lg = grid(cfg["l_min"], cfg["l_max"], cfg["step"])
    counts = np.array([int(np.sum(rf[neg] <= L)) for L in lg], dtype=np.int64)
    kl = int(np.argmin(np.abs(counts - cnt_ref)))      # first minimum
    l_star = float(lg[kl])
    out["l_star"] = l_star
    out["l_new"] = smooth_update(l_old, l_star, cfg["delta_l"])
    out["l_updated"] = True

    # upper bound: match the positive-to-negative update ratio at L*
    if rho_ref is None:
        return out
    hg = grid(cfg["h_min"], cfg["h_max"], cfg["step"])
    rhos = [rho(a, w, pi, r_fp8, l_star, H)[0] for H in hg]
    if rhos[0] is None:                                 # no negative update left above L*
        return out
    dist = np.array([abs(v - rho_ref) for v in rhos])
    kh = int(np.argmin(dist))                           # first minimum
    out["h_star"] = float(hg[kh])
    out["rho_fp8"] = rhos[kh]
    out["h_new"] = smooth_update(h_old, out["h_star"], cfg["delta_h"])
    out["h_updated"] = True
    return out
