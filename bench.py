"""Throughput of the FP8 linear-layer hot path on one MI355X.

One step = quantize the activations X[16384, 4096] per 1x128 block, quantize
the weights W[12288, 4096] per 128x128 block, and run the blockwise scaled
FP8 GEMM Y = X W^T (8B-class FFN up-projection, one 16K-token sequence;
paper Sec. 2.2, Eq. 3, and the FP8 training engine of Sec. 5.3).  Inputs are
seeded synthetic bf16 tensors resident in HBM before timing starts.

Prints one JSON line: value = GEMM flops (2 M N K) per step time in TFLOP/s,
plus the roofline of the dominant kernel (the GEMM, timed with HIP events on
its stream) and the oracle's CPU throughput on a bounded sample.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_FP8_TFLOPS = 5000.0   # MI355X dense FP8 MFMA
PEAK_HBM_GBS = 8000.0      # MI355X HBM3E

WORKLOADS = {
    "8b_ffn_up_fwd_blockwise": (16384, 4096, 12288),
}


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=100)
    p.add_argument("--warmup", type=int, default=50,
                   help="untimed steps first (the clock settles over the first few dozen)")
    p.add_argument("--workload", default="8b_ffn_up_fwd_blockwise", choices=sorted(WORKLOADS))
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-extras", action="store_true",
                   help="skip the timings of the kernels outside the step (backward-pass quantizer)")
    p.add_argument("--cpu-rows", type=int, default=2048,
                   help="rows of Y the oracle's exact GEMM computes for the CPU baseline")
    p.add_argument("--sweep", action="store_true",
                   help="instead of the step's line: one JSON line per FFN up-projection shape of "
                        "the 8B, 14B and 32B models at 4096, 8192 and 16384 tokens")
    p.add_argument("--config", type=int, choices=(1, 2, 3, 4, 5), default=None,
                   help="instead of the step's line: one JSON line per quantizer and GEMM of one "
                        "of the five workloads (1 tiny per-tensor, 2 8B blockwise forward, 3 8B "
                        "rowwise, 4 decode, 5 32B training layers), each its median over timed "
                        "repetitions, with the last-level cache flushed before each repetition of "
                        "the HBM-bound kernels")
    p.add_argument("--reps", type=int, default=50, help="timed repetitions per kernel with --config")
    p.add_argument("--settle-s", type=float, default=1.0,
                   help="seconds of untimed steps before the warmup steps, so that the timed "
                        "steps run at the clock the GPU holds under this load")
    p.add_argument("--calibrate-copy-mib", type=int, default=0,
                   help="after timing, run one plain device-to-device copy of this many "
                        "MiB: a kernel of known traffic to scale HBM byte counters by")
    return p.parse_args()


# Kernel sources whose change invalidates recorded HBM counters.
GEMM_SOURCES = ["paper_2609_22870_amd/csrc/gemm.hip", "paper_2609_22870_amd/csrc/device_common.h",
                "paper_2609_22870_amd/csrc/internal.h", "paper_2609_22870_amd/_build.py"]


def sources_digest(paths):
    import hashlib
    h = hashlib.sha256()
    for p in paths:
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def recorded_traffic(workload):
    """HBM bytes per GEMM launch from the committed rocprofv3 counter summary
    of this workload: FETCH_SIZE and WRITE_SIZE (KiB per dispatch), each
    multiplied by its copy-kernel calibration factor.  None when there is no
    summary or the GEMM sources changed since it was taken."""
    path = os.path.join(ROOT, "profiles", "gemm_%s_counters.md" % workload)
    if not os.path.exists(path):
        return None
    rec = {}
    with open(path) as f:
        for line in f:
            if line.startswith("    ") and ": " in line:
                k, v = line.strip().split(": ", 1)
                rec[k] = v
    try:
        if rec["gemm_sources_sha256"] != sources_digest(GEMM_SOURCES):
            return None
        return (float(rec["gemm_fetch_kib"]) * float(rec["fetch_factor"]) +
                float(rec["gemm_write_kib"]) * float(rec["write_factor"])) * 1024.0
    except (KeyError, ValueError):
        return None


def host_cpu():
    """nproc, the cores this process may use and the CPU model name."""
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"nproc": os.cpu_count(), "affinity_cores": len(os.sched_getaffinity(0)), "cpu_model": model}


def cpu_baseline(x, w, M, K, N, rows):
    """The oracle (untuned) on the host cores:
    * quantizers on the full tensors of the step: X [M, K] per 1x128 block
      and W [N, K] per 128x128 block, on one thread and on all cores (the
      rows split into contiguous chunks of whole units, one oracle call per
      chunk; the oracle's ctypes calls release the GIL);
    * the exact GEMM on `rows` rows of Y spread over all of M, on all cores,
      and its time for all M rows extrapolated from them (labelled so).
    value: the step's flops over the all-core step time (both quantizers on
    the full tensors plus the extrapolated GEMM)."""
    from concurrent.futures import ThreadPoolExecutor

    import numpy as np

    import oracle
    from paper_2609_22870_amd import synth

    cores = max(1, min(16, len(os.sched_getaffinity(0))))
    xs = synth.bf16_bits(x)
    wb = synth.bf16_bits(w)
    qbytes = lambda r, c, n_scales: 3.0 * r * c + 4.0 * n_scales

    t0 = time.perf_counter()
    ox, osx = oracle.quantize(xs, oracle.BLOCK_1x128)
    tx1 = time.perf_counter() - t0
    t0 = time.perf_counter()
    ow, osw = oracle.quantize(wb, oracle.BLOCK_128x128)
    tw1 = time.perf_counter() - t0

    def chunks(n_rows, unit):
        b = np.linspace(0, n_rows // unit, 4 * cores + 1).astype(np.int64) * unit
        return [(int(a), int(c)) for a, c in zip(b[:-1], b[1:]) if c > a]

    with ThreadPoolExecutor(cores) as ex:
        t0 = time.perf_counter()
        list(ex.map(lambda ab: oracle.quantize(xs[ab[0]:ab[1]], oracle.BLOCK_1x128), chunks(M, 1)))
        txn = time.perf_counter() - t0
        t0 = time.perf_counter()
        list(ex.map(lambda ab: oracle.quantize(wb[ab[0]:ab[1]], oracle.BLOCK_128x128), chunks(N, 128)))
        twn = time.perf_counter() - t0
        sample = np.linspace(0, M - 1, rows).astype(np.int64)
        t0 = time.perf_counter()
        list(ex.map(lambda r: oracle.gemm_rows(ox, osx, oracle.BLOCK_1x128, ow, osw, oracle.BLOCK_128x128, r),
                    np.array_split(sample, 4 * cores)))
        tg = time.perf_counter() - t0
    tg_full = tg * M / rows
    flops = 2.0 * M * N * K
    xb, wbytes = qbytes(M, K, osx.size), qbytes(N, K, osw.size)
    out = {
        "value": flops / (txn + twn + tg_full) / 1e12,
        "unit": "TFLOP/s",
        "cores": cores,
        "kind": "oracle",
        "sample": "quantizers on the full X [%d, %d] (1x128) and W [%d, %d] (128x128); exact "
                  "int64/binary128 GEMM on %d of %d rows of Y = X W^T spread over M, its full "
                  "time extrapolated; value = 2MNK over the all-core quantizers plus the "
                  "extrapolated GEMM" % (M, K, N, K, rows, M),
        "quantize_x_1x128": {"one_thread_s": round(tx1, 3), "one_thread_gbs": round(xb / tx1 / 1e9, 3),
                             "all_cores_s": round(txn, 3), "all_cores_gbs": round(xb / txn / 1e9, 3),
                             "elements_per_s_all_cores": round(M * K / txn)},
        "quantize_w_128x128": {"one_thread_s": round(tw1, 3), "one_thread_gbs": round(wbytes / tw1 / 1e9, 3),
                               "all_cores_s": round(twn, 3), "all_cores_gbs": round(wbytes / twn / 1e9, 3),
                               "elements_per_s_all_cores": round(N * K / twn)},
        "gemm_sample_rows": rows,
        "gemm_sample_s": round(tg, 3),
        "gemm_mac_per_s": round(rows * N * K / tg),
        "gemm_full_extrapolated_s": round(tg_full, 1),
    }
    out.update(host_cpu())
    return out


def time_extras(torch, fp8q, synth, dev, x, w, xq, sx, wq, sw, reps=20):
    """Kernels next to the step, each timed alone with HIP events on the
    launch stream:
    * the dual-layout quantizer of the backward pass on the 32B FFN output
      gradient dY[16384, 25600] (its 1x128 codes for dgrad and its
      transposed 128x1 codes for wgrad from one read), against the two
      single-layout calls it replaces;
    * the step's GEMM with its output quantized per 1x128 block in the
      epilogue (the next layer's activation operand), against the GEMM
      followed by the quantizer on its bf16 output;
    * Calibrated Clipping (Alg. 1) over one batch of the paper's GRPO setup
      (256 prompts x 8 responses of 512-8192 tokens: 8.9 M tokens, five
      float32 arrays), both of its kernels;
    * the step's GEMM on operands quantized with power-of-two scales (a
      variant, not the paper's scale), whose block scales enter the matrix
      instruction, with that quantization of X;
    * the E5M2 variant for gradients on the same dY: its dual-layout
      quantization, and the 32B up-projection's data-gradient GEMM dX = dY W
      (16384 x 25600 -> 5120) with dY's codes in E5M2 against E4M3;
    * the grouped GEMM of the fused projections of the step's X (query, key
      and value: 4096 + 1024 + 1024 outputs; gate and up: 2 x 12288) in one
      launch, against one fp8q_gemm call per projection;
    * the paper's three scaling recipes on the step's layer (tensorwise,
      rowwise: per-token X and per-output-channel W, blockwise): quantize X,
      quantize W and the GEMM, each timed."""
    rows, cols = 16384, 25600
    dy = synth.grads(rows, cols, seed=synth.seed_for(5, 2), device=dev)
    outs = fp8q.quantize_dual(dy)
    r1 = fp8q.quantize(dy, fp8q.BLOCK_1x128)
    r2 = fp8q.quantize(dy, fp8q.BLOCK_128x1, transposed=True)
    stream = torch.cuda.current_stream(dev)

    def timed(f):
        for _ in range(3):
            f()
        s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        s.record(stream)
        for _ in range(reps):
            f()
        e.record(stream)
        torch.cuda.synchronize()
        return s.elapsed_time(e) / reps * 1000.0

    t_dual = timed(lambda: fp8q.quantize_dual(dy, *outs))
    t_two = timed(lambda: (fp8q.quantize(dy, fp8q.BLOCK_1x128, codes=r1[0], scales=r1[1]),
                           fp8q.quantize(dy, fp8q.BLOCK_128x1, transposed=True, codes=r2[0], scales=r2[1])))
    nbytes = 4.0 * rows * cols + 4.0 * (outs[1].numel() + outs[3].numel())
    gbs = nbytes / (t_dual * 1e-6) / 1e9
    del r1, r2

    k_in = 5120
    w32 = synth.weights(cols, k_in, seed=synth.seed_for(5, 1), device=dev)
    wt, swt = fp8q.quantize(w32, fp8q.BLOCK_128x128, transposed=True)    # W^T [5120, 25600]
    del w32
    outs5 = fp8q.quantize_dual(dy, e5m2=True)
    t_dual5 = timed(lambda: fp8q.quantize_dual(dy, *outs5, e5m2=True))
    dx = torch.empty((rows, k_in), dtype=torch.bfloat16, device=dev)
    t_dg4 = timed(lambda: fp8q.gemm(outs[0], outs[1], fp8q.BLOCK_1x128, wt, swt, fp8q.BLOCK_128x128, out=dx))
    t_dg5 = timed(lambda: fp8q.gemm_formats(outs5[0], outs5[1], fp8q.BLOCK_1x128, wt, swt, fp8q.BLOCK_128x128,
                                            fp8q.A_E5M2, out=dx))
    dg_flops = 2.0 * rows * cols * k_in
    del dy, outs, outs5, wt, swt, dx

    M, N, K = xq.shape[0], wq.shape[0], xq.shape[1]
    y = torch.empty((M, N), dtype=torch.bfloat16, device=dev)
    yq = torch.empty((M, N), dtype=torch.uint8, device=dev)
    ys = torch.empty(fp8q.scales_count(M, N, fp8q.BLOCK_1x128), dtype=torch.float32, device=dev)
    t_fused = timed(lambda: fp8q.gemm_quantized(xq, sx, fp8q.BLOCK_1x128, wq, sw, fp8q.BLOCK_128x128,
                                                codes=yq, scales=ys))
    t_sep = timed(lambda: (fp8q.gemm(xq, sx, fp8q.BLOCK_1x128, wq, sw, fp8q.BLOCK_128x128, out=y),
                           fp8q.quantize(y, fp8q.BLOCK_1x128, codes=yq, scales=ys)))
    tflops = 2.0 * M * N * K / (t_fused * 1e-6) / 1e12
    del yq, ys

    xb = torch.empty_like(xq)
    sxb = torch.empty_like(sx)
    wb, swb = fp8q.quantize(w, fp8q.BLOCK_128x128, pow2=True)
    t_qx2 = timed(lambda: fp8q.quantize(x, fp8q.BLOCK_1x128, codes=xb, scales=sxb, pow2=True))
    t_pow2 = timed(lambda: fp8q.gemm_pow2(xb, sxb, fp8q.BLOCK_1x128, wb, swb, fp8q.BLOCK_128x128, out=y))
    pow2_tflops = 2.0 * M * N * K / (t_pow2 * 1e-6) / 1e12
    del y, xb, sxb, wb, swb

    # the paper's three scaling recipes on the step's layer: quantize X,
    # quantize W, GEMM
    recipes = {}
    for name, gx, gw in (("tensorwise", fp8q.TENSOR, fp8q.TENSOR), ("rowwise", fp8q.ROW, fp8q.ROW),
                         ("blockwise", fp8q.BLOCK_1x128, fp8q.BLOCK_128x128)):
        xa, sxa = fp8q.quantize(x, gx)
        wa, swa = fp8q.quantize(w, gw)
        ya = torch.empty((M, N), dtype=torch.bfloat16, device=dev)
        t_x = timed(lambda: fp8q.quantize(x, gx, codes=xa, scales=sxa))
        t_w = timed(lambda: fp8q.quantize(w, gw, codes=wa, scales=swa))
        t_g = timed(lambda: fp8q.gemm(xa, sxa, gx, wa, swa, gw, out=ya))
        step = t_x + t_w + t_g
        recipes[name] = {"quantize_x_us": round(t_x, 1), "quantize_w_us": round(t_w, 1), "gemm_us": round(t_g, 1),
                         "step_us": round(step, 1),
                         "step_tflops": round(2.0 * M * N * K / (step * 1e-6) / 1e12, 1),
                         "gemm_tflops": round(2.0 * M * N * K / (t_g * 1e-6) / 1e12, 1)}
        del xa, sxa, wa, swa, ya

    grouped = {}
    for kind, widths in (("qkv", (4096, 1024, 1024)), ("gate_up", (12288, 12288))):
        probs = []
        for i, n in enumerate(widths):
            wq_i, sw_i = fp8q.quantize(synth.weights(n, K, seed=synth.seed_for(6, 1, i), device=dev),
                                       fp8q.BLOCK_128x128)
            probs.append((xq, sx, wq_i, sw_i))
        outs = fp8q.gemm_grouped(probs, fp8q.BLOCK_1x128, fp8q.BLOCK_128x128)
        t_grp = timed(lambda: fp8q.gemm_grouped(probs, fp8q.BLOCK_1x128, fp8q.BLOCK_128x128, outs=outs))
        t_calls = timed(lambda: [fp8q.gemm(a, sa, fp8q.BLOCK_1x128, b, sb, fp8q.BLOCK_128x128, out=c)
                                 for (a, sa, b, sb), c in zip(probs, outs)])
        flops = 2.0 * M * K * sum(widths)
        grouped[kind] = {"widths": list(widths), "us": round(t_grp, 1),
                         "tflops": round(flops / (t_grp * 1e-6) / 1e12, 1),
                         "separate_calls_us": round(t_calls, 1)}
        del probs, outs

    rl = {k: v.to(dev) for k, v in synth.rl_batch(**synth.RL_BATCH, seed=5001).items()}
    keys = ("adv", "w_tis", "pi_sampler", "r_bf16", "r_fp8")
    ntok = rl["adv"].numel()
    ws = torch.empty(fp8q.lib().fp8q_calibrate_clip_workspace(ntok), dtype=torch.uint8, device=dev)
    res = torch.empty(80, dtype=torch.uint8, device=dev)
    t_clip = timed(lambda: fp8q.calibrate_clip(*(rl[k] for k in keys), 0.6, 1.8, workspace=ws,
                                               result=res, read=False))
    clip_bytes = 20.0 * ntok
    clip_gbs = clip_bytes / (t_clip * 1e-6) / 1e9
    return {"quantize_dual_32b_dy": {
        "shape": [rows, cols], "us": round(t_dual, 1), "gbs": round(gbs, 1),
        "frac_hbm": round(gbs / PEAK_HBM_GBS, 4),
        "algorithmic_bytes": round(nbytes), "two_single_layout_calls_us": round(t_two, 1)},
        "gemm_quantized_output_8b_ffn_up": {
        "shape": [M, K, N], "us": round(t_fused, 1), "tflops": round(tflops, 1),
        "frac_mfma": round(tflops / PEAK_FP8_TFLOPS, 4),
        "gemm_then_quantize_us": round(t_sep, 1)},
        "gemm_pow2_scales_8b_ffn_up": {
        "shape": [M, K, N], "us": round(t_pow2, 1), "tflops": round(pow2_tflops, 1),
        "frac_mfma": round(pow2_tflops / PEAK_FP8_TFLOPS, 4), "quantize_x_pow2_us": round(t_qx2, 1)},
        "e5m2_dy_32b_up": {
        "dual_quantize_us": round(t_dual5, 1), "dgrad_shape": [rows, cols, k_in],
        "dgrad_e5m2_us": round(t_dg5, 1), "dgrad_e5m2_tflops": round(dg_flops / (t_dg5 * 1e-6) / 1e12, 1),
        "dgrad_e4m3_us": round(t_dg4, 1), "dgrad_e4m3_tflops": round(dg_flops / (t_dg4 * 1e-6) / 1e12, 1)},
        "gemm_grouped_8b_fused_projections": grouped,
        "scaling_recipes_8b_ffn_up": recipes,
        "calibrated_clipping_grpo_batch": {
        "tokens": ntok, "us": round(t_clip, 1), "gbs": round(clip_gbs, 1),
        "frac_hbm": round(clip_gbs / PEAK_HBM_GBS, 4), "algorithmic_bytes": round(clip_bytes)}}


def clock_under_load(torch, f, seconds=1.0):
    """Shader clock and socket power while f (one GEMM launch) runs back to
    back for about `seconds`, sampled every 10 ms from the GPU metrics table
    through amdsmi in a second thread; with the GEMM's event-timed average
    over the same period.  None when amdsmi is not importable or the device
    is not found."""
    import threading
    try:
        import amdsmi
        amdsmi.amdsmi_init()
    except Exception as e:  # the metric is optional: report why it is missing
        return {"error": "amdsmi: %s" % e}
    try:
        handles = amdsmi.amdsmi_get_processor_handles()
        h = handles[0] if len(handles) == 1 else None
        if h is None:
            bus = getattr(torch.cuda.get_device_properties(0), "pci_bus_id", None)
            for c in handles:
                if bus is not None and int(amdsmi.amdsmi_get_gpu_device_bdf(c).split(":")[1], 16) == bus:
                    h = c
        if h is None:
            return {"error": "device not matched among %d" % len(handles)}
        clocks, power, stop = [], [], threading.Event()

        def poll():
            while not stop.is_set():
                m = amdsmi.amdsmi_get_gpu_metrics_info(h)
                xcd = [v for v in m.get("current_gfxclks", []) if isinstance(v, int) and 0 < v < 10000]
                if xcd:
                    clocks.append(sum(xcd) / len(xcd))
                p = m.get("current_socket_power")
                if isinstance(p, (int, float)) and 0 < p < 5000:
                    power.append(float(p))
                stop.wait(0.01)

        th = threading.Thread(target=poll, daemon=True)
        s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        th.start()
        t0, n = time.perf_counter(), 0
        s.record()
        while time.perf_counter() - t0 < seconds:
            for _ in range(10):
                f()
            n += 10
            torch.cuda.synchronize()
        e.record()
        torch.cuda.synchronize()
        stop.set()
        th.join()
        med = lambda v: sorted(v)[len(v) // 2] if v else None
        return {"gfx_mhz_median": med(clocks), "gfx_mhz_min": min(clocks) if clocks else None,
                "gfx_mhz_max": max(clocks) if clocks else None, "socket_power_w_median": med(power),
                "samples": len(clocks), "gemm_us": round(s.elapsed_time(e) / n * 1000.0, 1), "launches": n}
    except Exception as e:
        return {"error": "amdsmi: %s" % e}
    finally:
        try:
            amdsmi.amdsmi_shut_down()
        except Exception:
            pass


# FFN up-projection (hidden K -> intermediate N) of the model sizes the
# paper's throughput comparison covers (Sec. 5.3): Qwen3-8B, Qwen3-14B, and
# the 32B width used throughout (25600); token counts of 4K, 8K and 16K.
SWEEP_MODELS = (("8b", 4096, 12288), ("14b", 5120, 17408), ("32b", 5120, 25600))
SWEEP_TOKENS = (4096, 8192, 16384)


def run_sweep(torch, fp8q, synth, dev, warmup=10, reps=30):
    """The step (quantize X per 1x128, quantize W per 128x128, blockwise
    GEMM) at each sweep shape, every kernel bracketed by HIP events as in
    the main timing; one JSON line per shape."""
    stream = torch.cuda.current_stream(dev)
    for mi, (name, K, N) in enumerate(SWEEP_MODELS):
        w = synth.weights(N, K, seed=synth.seed_for(10 + mi, 1), device=dev)
        wq = torch.empty((N, K), dtype=torch.uint8, device=dev)
        sw = torch.empty(fp8q.scales_count(N, K, fp8q.BLOCK_128x128), dtype=torch.float32, device=dev)
        for M in SWEEP_TOKENS:
            x = synth.activations(M, K, seed=synth.seed_for(10 + mi, 0), outlier_seed=synth.seed_for(10 + mi, 3),
                                  device=dev)
            xq = torch.empty((M, K), dtype=torch.uint8, device=dev)
            sx = torch.empty(fp8q.scales_count(M, K, fp8q.BLOCK_1x128), dtype=torch.float32, device=dev)
            y = torch.empty((M, N), dtype=torch.bfloat16, device=dev)

            def step(ev=None):
                if ev is not None:
                    ev[0].record(stream)
                fp8q.quantize(x, fp8q.BLOCK_1x128, codes=xq, scales=sx)
                if ev is not None:
                    ev[1].record(stream)
                fp8q.quantize(w, fp8q.BLOCK_128x128, codes=wq, scales=sw)
                if ev is not None:
                    ev[2].record(stream)
                fp8q.gemm(xq, sx, fp8q.BLOCK_1x128, wq, sw, fp8q.BLOCK_128x128, out=y)
                if ev is not None:
                    ev[3].record(stream)

            for _ in range(warmup):
                step()
            events = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(reps)]
            for ev in events:
                step(ev)
            torch.cuda.synchronize()
            avg = lambda a, b: sum(e[a].elapsed_time(e[b]) for e in events) / reps * 1000.0
            t_qx, t_qw, t_g = avg(0, 1), avg(1, 2), avg(2, 3)
            flops = 2.0 * M * N * K
            print(json.dumps({
                "sweep": "%s_ffn_up_fwd_blockwise" % name, "M": M, "K": K, "N": N,
                "gemm_us": round(t_g, 1), "gemm_tflops": round(flops / t_g * 1e-6, 1),
                "gemm_frac_fp8_peak": round(flops / t_g * 1e-6 / PEAK_FP8_TFLOPS, 4),
                "quantize_x_us": round(t_qx, 1), "quantize_w_us": round(t_qw, 1),
                "step_us": round(t_qx + t_qw + t_g, 1),
                "step_tflops": round(flops / (t_qx + t_qw + t_g) * 1e-6, 1)}), flush=True)
            del x, xq, sx, y
        del w, wq, sw


class Flush:
    """A read of 1 GiB (a max over a float32 buffer: four times the 256 MB
    last-level cache) run before a repetition, outside its events, so that
    the kernel timed next reads its operands from HBM.  Read-only: a flush
    that writes leaves dirty lines whose write-back would land on the timed
    kernel."""

    def __init__(self, torch, dev):
        self.buf = torch.zeros(256 << 20, dtype=torch.float32, device=dev)
        self.out = torch.empty((), dtype=torch.float32, device=dev)

    def __call__(self):
        torch_amax(self.buf, self.out)


def torch_amax(buf, out):
    import torch
    torch.amax(buf, dim=0, out=out)


def time_op(torch, stream, f, reps, warmup=10, flush=None):
    """Sorted durations in us of `reps` calls of f, each bracketed by HIP
    events on the launch stream, after `warmup` untimed calls; with flush,
    flush() runs before every call, outside the events."""
    for _ in range(warmup):
        if flush is not None:
            flush()
        f()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
    for s, e in evs:
        if flush is not None:
            flush()
        s.record(stream)
        f()
        e.record(stream)
    torch.cuda.synchronize()
    return sorted(s.elapsed_time(e) * 1000.0 for s, e in evs)


def time_rotated(torch, stream, fs, reps, warmup=3, flush=None):
    """Sorted per-call durations in us: each repetition runs every f of fs
    back to back between two HIP events on the launch stream (after
    flush(), outside the events), and counts the elapsed time over
    len(fs).  The fs work on distinct buffers that together exceed the
    last-level cache, so each call finds its operands in HBM, and the
    launch gaps of a single timed call are spread over the group."""
    for _ in range(warmup):
        if flush is not None:
            flush()
        for f in fs:
            f()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
    for s, e in evs:
        if flush is not None:
            flush()
        s.record(stream)
        for f in fs:
            f()
        e.record(stream)
    torch.cuda.synchronize()
    return sorted(s.elapsed_time(e) * 1000.0 / len(fs) for s, e in evs)


def rotation(nbytes, total=768 << 20, most=16):
    """How many buffer sets of nbytes each make up about `total` bytes (at
    least 2, at most `most`)."""
    return int(max(2, min(most, -(-total // max(1, int(nbytes))))))


def percentiles(ts):
    n = len(ts)
    return ts[min(n - 1, int(0.1 * n))], ts[n // 2], ts[min(n - 1, int(0.9 * n))]


GRAN_NAMES = {0: "tensor", 1: "row", 2: "col", 3: "1x128", 4: "128x1", 5: "128x128"}


def run_config(torch, fp8q, synth, dev, cfg, reps):
    """One JSON line per quantizer and GEMM of workload `cfg` (the five
    workloads of the parity tests, at full size), each the median and
    p10 / p90 over `reps` event-timed repetitions after 10 untimed ones.
    Quantizers and the HBM-bound decode GEMMs run with the last-level cache
    flushed before every repetition; the MFMA-bound GEMMs back to back.
    Rates: quantizer bytes are 2 (bf16 read) + 1 per code written + 4 per
    scale; GEMM bytes MK + NK + 2MN + 4 per scale; GEMM work 2MNK flops."""
    stream = torch.cuda.current_stream(dev)
    flush = Flush(torch, dev)
    names = {1: "tiny_tensorwise", 2: "8b_ffn_up_fwd_blockwise", 3: "8b_rowwise", 4: "8b_decode_blockwise",
             5: "32b_train_blockwise"}

    def emit(op, ts, bound, work, unit_peak, extra):
        p10, p50, p90 = percentiles(ts)
        line = {"config": cfg, "workload": names[cfg], "op": op, "us_p50": round(p50, 2),
                "us_p10": round(p10, 2), "us_p90": round(p90, 2), "reps": len(ts), "bound": bound}
        if bound == "hbm":
            rate = work / (p50 * 1e-6) / 1e9
            line.update({"gbs": round(rate, 1), "frac_hbm": round(rate / PEAK_HBM_GBS, 4),
                         "algorithmic_bytes": round(work)})
        elif bound == "mfma":
            rate = work / (p50 * 1e-6) / 1e12
            line.update({"tflops": round(rate, 1), "frac_fp8_peak": round(rate / PEAK_FP8_TFLOPS, 4),
                         "flops": round(work)})
        else:
            line.update({"flops": round(work)})
        line.update(extra)
        print(json.dumps(line), flush=True)

    def quant(label, x, g, transposed=False, **kw):
        codes, scales = fp8q.quantize(x, g, transposed, **kw)
        rows, cols = x.shape
        nbytes = 3.0 * rows * cols + 4.0 * scales.numel()
        sets = [(x, codes, scales)] + [(x.clone(), torch.empty_like(codes), torch.empty_like(scales))
                                       for _ in range(rotation(nbytes) - 1)]
        fs = [lambda s=s: fp8q.quantize(s[0], g, transposed, codes=s[1], scales=s[2], **kw) for s in sets]
        ts = time_rotated(torch, stream, fs, reps, flush=flush)
        del sets, fs
        emit("quantize " + label, ts, "hbm", nbytes, PEAK_HBM_GBS,
             {"shape": [rows, cols], "granularity": GRAN_NAMES[g], "transposed": transposed, "flushed": True})
        return codes, scales

    def dual(label, x):
        outs = fp8q.quantize_dual(x)
        rows, cols = x.shape
        nbytes = 4.0 * rows * cols + 4.0 * (outs[1].numel() + outs[3].numel())
        sets = [(x, outs)] + [(x.clone(), tuple(torch.empty_like(o) for o in outs))
                              for _ in range(rotation(nbytes) - 1)]
        fs = [lambda s=s: fp8q.quantize_dual(s[0], *s[1]) for s in sets]
        ts = time_rotated(torch, stream, fs, reps, flush=flush)
        del sets, fs
        emit("quantize_dual " + label, ts, "hbm", nbytes, PEAK_HBM_GBS,
             {"shape": [rows, cols], "granularity": "1x128 + 128x1 transposed", "flushed": True})
        return outs

    def gemm(label, a, sa, ga, b, sb, gb, hbm=False, splitk=False):
        """splitk: fp8q_gemm_splitk (one zero-filled workspace shared by
        the calls, which run in order on one stream) instead of fp8q_gemm."""
        M, K = a.shape
        N = b.shape[0]
        out = torch.empty((M, N), dtype=torch.bfloat16, device=dev)
        if splitk:
            ws = torch.zeros(max(fp8q.gemm_splitk_workspace(M, N, K), 16), dtype=torch.uint8, device=dev)
            call = lambda a_, b_, o_: fp8q.gemm_splitk(a_, sa, ga, b_, sb, gb, out=o_, workspace=ws)
        else:
            call = lambda a_, b_, o_: fp8q.gemm(a_, sa, ga, b_, sb, gb, out=o_)
        f = lambda: call(a, b, out)
        flops = 2.0 * M * N * K
        nbytes = 1.0 * M * K + 1.0 * N * K + 2.0 * M * N + 4.0 * (sa.numel() + sb.numel())
        extra = {"shape_mkn": [M, K, N], "scaling": "%s x %s" % (GRAN_NAMES[ga], GRAN_NAMES[gb]),
                 "flushed": hbm}
        if hbm:
            # distinct copies of both operands (and outputs) for every call
            sets = [(a, b, out)] + [(a.clone(), b.clone(), torch.empty_like(out))
                                    for _ in range(rotation(nbytes) - 1)]
            fs = [lambda s=s: call(s[0], s[1], s[2]) for s in sets]
            ts = time_rotated(torch, stream, fs, reps, flush=flush)
            del sets, fs
            warm = percentiles(time_op(torch, stream, f, reps))[1]
            extra["tflops_at_p50"] = round(flops / (percentiles(ts)[1] * 1e-6) / 1e12, 1)
            extra["us_p50_back_to_back"] = round(warm, 2)
            emit(("gemm_splitk " if splitk else "gemm ") + label, ts, "hbm", nbytes, PEAK_HBM_GBS, extra)
        elif cfg == 1:
            emit("gemm " + label, time_op(torch, stream, f, reps), "launch", flops, None, extra)
        else:
            extra["algorithmic_bytes"] = round(nbytes)
            emit("gemm " + label, time_op(torch, stream, f, reps), "mfma", flops, PEAK_FP8_TFLOPS, extra)
        del out

    if cfg == 1:
        a = synth.normal_bf16((128, 256), 1.0, synth.seed_for(1, 0), dev)
        b = synth.normal_bf16((256, 256), 0.02, synth.seed_for(1, 1), dev)
        A, sA = quant("A", a, fp8q.TENSOR)
        B, sB = quant("B", b, fp8q.TENSOR)
        gemm("tiny", A, sA, fp8q.TENSOR, B, sB, fp8q.TENSOR)
    elif cfg == 2:
        M, K, N = synth.WORKLOADS["8b_ffn_up_fwd_blockwise"]["shapes"][0]
        x = synth.activations(M, K, seed=synth.seed_for(2, 0), outlier_seed=synth.seed_for(2, 3), device=dev)
        w = synth.weights(N, K, seed=synth.seed_for(2, 1), device=dev)
        X, sX = quant("X", x, fp8q.BLOCK_1x128)
        W, sW = quant("W", w, fp8q.BLOCK_128x128)
        gemm("fwd", X, sX, fp8q.BLOCK_1x128, W, sW, fp8q.BLOCK_128x128)
    elif cfg in (3, 4):
        key = "8b_rowwise" if cfg == 3 else "8b_decode_blockwise"
        gx, gw = (fp8q.ROW, fp8q.ROW) if cfg == 3 else (fp8q.BLOCK_1x128, fp8q.BLOCK_128x128)
        for i, (M, K, N) in enumerate(synth.WORKLOADS[key]["shapes"]):
            x = synth.activations(M, K, seed=synth.seed_for(cfg, 0, i), outlier_seed=synth.seed_for(cfg, 3, i),
                                  device=dev)
            w = synth.weights(N, K, seed=synth.seed_for(cfg, 1, i), device=dev)
            tag = "%dx%dx%d" % (M, K, N)
            X, sX = quant("X " + tag, x, gx)
            W, sW = quant("W " + tag, w, gw)
            gemm(tag, X, sX, gx, W, sW, gw, hbm=(cfg == 4))
            if cfg == 4 and fp8q.gemm_splitk_workspace(M, N, K) > 0:
                gemm(tag, X, sX, gx, W, sW, gw, hbm=True, splitk=True)
            del x, w, X, sX, W, sW
    else:
        T = 16384
        for si, proj, k_in, n_out in ((0, "up", 5120, 25600), (3, "down", 25600, 5120)):
            x = synth.activations(T, k_in, seed=synth.seed_for(5, 0, si), outlier_seed=synth.seed_for(5, 3, si),
                                  device=dev)
            w = synth.weights(n_out, k_in, seed=synth.seed_for(5, 1, si), device=dev)
            dy = synth.grads(T, n_out, seed=synth.seed_for(5, 2, si), device=dev)
            X, sX = quant(proj + " X (fwd)", x, fp8q.BLOCK_1x128)
            W, sW = quant(proj + " W (fwd)", w, fp8q.BLOCK_128x128)
            Wt, sWt = quant(proj + " W^T (dgrad)", w, fp8q.BLOCK_128x128, transposed=True)
            dY, sdY, dYt, sdYt = dual(proj + " dY (dgrad, wgrad)", dy)
            Xt, sXt = quant(proj + " X^T (wgrad)", x, fp8q.BLOCK_128x1, transposed=True)
            gemm(proj + " fwd", X, sX, fp8q.BLOCK_1x128, W, sW, fp8q.BLOCK_128x128)
            del X, sX, W, sW
            gemm(proj + " dgrad", dY, sdY, fp8q.BLOCK_1x128, Wt, sWt, fp8q.BLOCK_128x128)
            del dY, sdY, Wt, sWt
            gemm(proj + " wgrad", Xt, sXt, fp8q.BLOCK_1x128, dYt, sdYt, fp8q.BLOCK_1x128)
            del x, w, dy, Xt, sXt, dYt, sdYt


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py runs on one GPU only: this build has no multi-GPU path "
              "(--gpus %d requested)" % args.gpus, file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2609_22870_amd as fp8q
    from paper_2609_22870_amd import synth

    M, K, N = WORKLOADS[args.workload]
    dev = torch.device("cuda:0")
    if args.sweep:
        run_sweep(torch, fp8q, synth, dev)
        return
    if args.config is not None:
        run_config(torch, fp8q, synth, dev, args.config, args.reps)
        return
    x = synth.activations(M, K, seed=synth.seed_for(2, 0), outlier_seed=synth.seed_for(2, 3), device=dev)
    w = synth.weights(N, K, seed=synth.seed_for(2, 1), device=dev)
    xq = torch.empty((M, K), dtype=torch.uint8, device=dev)
    wq = torch.empty((N, K), dtype=torch.uint8, device=dev)
    sx = torch.empty(fp8q.scales_count(M, K, fp8q.BLOCK_1x128), dtype=torch.float32, device=dev)
    sw = torch.empty(fp8q.scales_count(N, K, fp8q.BLOCK_128x128), dtype=torch.float32, device=dev)
    y = torch.empty((M, N), dtype=torch.bfloat16, device=dev)
    stream = torch.cuda.current_stream(dev)

    def step(ev=None):
        if ev is not None:
            ev[0].record(stream)
        fp8q.quantize(x, fp8q.BLOCK_1x128, codes=xq, scales=sx)
        if ev is not None:
            ev[1].record(stream)
        fp8q.quantize(w, fp8q.BLOCK_128x128, codes=wq, scales=sw)
        if ev is not None:
            ev[2].record(stream)
        fp8q.gemm(xq, sx, fp8q.BLOCK_1x128, wq, sw, fp8q.BLOCK_128x128, out=y)
        if ev is not None:
            ev[3].record(stream)

    # untimed steps for --settle-s seconds first: the shader clock ramps and
    # then settles under the power limit over the first tens of milliseconds
    # of load, so the timed steps run at the clock this load holds
    settle_steps = 0
    t_settle = time.perf_counter()
    while time.perf_counter() - t_settle < args.settle_s:
        for _ in range(10):
            step()
        settle_steps += 10
        torch.cuda.synchronize()
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    events = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    start.record(stream)
    for i in range(args.steps):
        step(events[i])
    end.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_step = start.elapsed_time(end) / args.steps

    qx_ms = sum(e[0].elapsed_time(e[1]) for e in events) / args.steps
    qw_ms = sum(e[1].elapsed_time(e[2]) for e in events) / args.steps
    gemm_ms = sum(e[2].elapsed_time(e[3]) for e in events) / args.steps
    gemm_sorted = sorted(e[2].elapsed_time(e[3]) for e in events)
    pct = lambda q: round(gemm_sorted[min(len(gemm_sorted) - 1, int(q * len(gemm_sorted)))] * 1000.0, 1)

    flops = 2.0 * M * N * K
    value = flops / (ms_step * 1e-3) / 1e12
    gemm_tflops = flops / (gemm_ms * 1e-3) / 1e12
    gemm_bytes = 1.0 * M * K + 1.0 * N * K + 2.0 * M * N + 4.0 * (M * (K // 128) + (N // 128) * (K // 128))
    traffic = recorded_traffic(args.workload)
    qx_bytes = 3.0 * M * K + 4.0 * M * (K // 128)
    qw_bytes = 3.0 * N * K + 4.0 * (N // 128) * (K // 128)
    out = {
        "metric": "FP8 blockwise GEMM TFLOP/s and % of dense FP8 MFMA peak, 8B-class shapes",
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "fp8_e4m3",
        "data": "synthetic",
        "config": {"workload": args.workload, "M": M, "K": K, "N": N,
                   "scaling": "1x128 activation blocks, 128x128 weight blocks",
                   "step": "quantize X + quantize W + blockwise FP8 GEMM"},
        "roofline": {"bound": "mfma", "achieved": round(gemm_tflops, 2),
                     "peak": PEAK_FP8_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(gemm_tflops / PEAK_FP8_TFLOPS, 4),
                     "traffic": None if traffic is None else round(traffic),
                     "algorithmic_bytes": round(gemm_bytes)},
        "pct_of_fp8_peak_step": round(100 * value / PEAK_FP8_TFLOPS, 2),
        "kernels_ms": {"quantize_x_1x128": round(qx_ms, 4), "quantize_w_128x128": round(qw_ms, 4),
                       "gemm_blockwise": round(gemm_ms, 4)},
        "quantize_gbs": {"x_1x128": round(qx_bytes / (qx_ms * 1e-3) / 1e9, 1),
                         "w_128x128": round(qw_bytes / (qw_ms * 1e-3) / 1e9, 1),
                         "hbm_peak": PEAK_HBM_GBS},
        "gemm_us_p10_p50_p90": [pct(0.1), pct(0.5), pct(0.9)],
        "timed_wall_s": round(wall, 3),
        "settle": {"seconds": args.settle_s, "untimed_steps": settle_steps},
    }
    # the quantizers alone, cold: each repetition quantizes distinct copies
    # of the input (together over the last-level cache) after a flush, so
    # that no operand comes from the caches (their in-step figures above may
    # find part of their input there): median over 50
    flush = Flush(torch, dev)

    def rotated(src, g, codes, scales, nbytes):
        sets = [(src, codes, scales)] + [(src.clone(), torch.empty_like(codes), torch.empty_like(scales))
                                         for _ in range(rotation(nbytes) - 1)]
        fs = [lambda s=s: fp8q.quantize(s[0], g, codes=s[1], scales=s[2]) for s in sets]
        return percentiles(time_rotated(torch, stream, fs, 50, flush=flush))[1]
    tqx = rotated(x, fp8q.BLOCK_1x128, xq, sx, qx_bytes)
    tqw = rotated(w, fp8q.BLOCK_128x128, wq, sw, qw_bytes)
    del flush
    out["quantize_flushed"] = {
        "x_1x128_us": round(tqx, 2), "x_1x128_gbs": round(qx_bytes / (tqx * 1e-6) / 1e9, 1),
        "x_1x128_frac_hbm": round(qx_bytes / (tqx * 1e-6) / 1e9 / PEAK_HBM_GBS, 4),
        "w_128x128_us": round(tqw, 2), "w_128x128_gbs": round(qw_bytes / (tqw * 1e-6) / 1e9, 1),
        "w_128x128_frac_hbm": round(qw_bytes / (tqw * 1e-6) / 1e9 / PEAK_HBM_GBS, 4)}
    # the shader clock the GEMM runs at: its peak at that clock is the
    # dense FP8 rate scaled by clock / 2400 MHz
    clk = clock_under_load(torch, lambda: fp8q.gemm(xq, sx, fp8q.BLOCK_1x128, wq, sw, fp8q.BLOCK_128x128, out=y))
    if clk and clk.get("gfx_mhz_median"):
        t = flops / (clk["gemm_us"] * 1e-6) / 1e12
        clk["gemm_tflops"] = round(t, 1)
        clk["frac_of_peak_at_this_clock"] = round(t / (PEAK_FP8_TFLOPS * clk["gfx_mhz_median"] / 2400.0), 4)
    out["clock_under_gemm"] = clk
    if args.calibrate_copy_mib > 0:
        n = args.calibrate_copy_mib << 20
        src = torch.zeros(n, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    if not args.no_extras:
        out["extra_kernels"] = time_extras(torch, fp8q, synth, dev, x, w, xq, sx, wq, sw)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(x.cpu(), w.cpu(), M, K, N, args.cpu_rows)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
