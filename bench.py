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
    p.add_argument("--cpu-rows", type=int, default=4096,
                   help="rows of X the oracle processes for the CPU baseline")
    p.add_argument("--sweep", action="store_true",
                   help="instead of the step's line: one JSON line per FFN up-projection shape of "
                        "the 8B, 14B and 32B models at 4096, 8192 and 16384 tokens")
    p.add_argument("--calibrate-copy-mib", type=int, default=0,
                   help="after timing, run one plain device-to-device copy of this many "
                        "MiB: a kernel of known traffic to scale HBM byte counters by")
    return p.parse_args()


# Kernel sources whose change invalidates recorded HBM counters.
GEMM_SOURCES = ["paper_2609_22870_amd/csrc/gemm.hip", "paper_2609_22870_amd/csrc/device_common.h",
                "paper_2609_22870_amd/csrc/internal.h"]


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


def cpu_baseline(x, w, M, K, N, rows):
    """The oracle (untuned) on a sample of the same step: `rows` rows of X
    quantized 1x128, the matching share of W's rows (rounded up to whole
    128-row blocks) quantized 128x128, and those rows of Y computed exactly.
    Runs on all host cores, one oracle call per thread."""
    from concurrent.futures import ThreadPoolExecutor

    import numpy as np

    import oracle
    from paper_2609_22870_amd import synth

    cores = max(1, min(16, len(os.sched_getaffinity(0))))
    xs = synth.bf16_bits(x[:rows])
    wrows = max(128, ((N * rows // M + 127) // 128) * 128)
    wb = synth.bf16_bits(w)
    t0 = time.perf_counter()
    with ThreadPoolExecutor(cores) as ex:
        xparts = np.array_split(np.arange(rows), cores)
        xres = list(ex.map(lambda r: oracle.quantize(xs[r[0]:r[-1] + 1], oracle.BLOCK_1x128), xparts))
        wblocks = [(i, min(wrows, i + 128)) for i in range(0, wrows, 128)]
        list(ex.map(lambda ab: oracle.quantize(wb[ab[0]:ab[1]], oracle.BLOCK_128x128), wblocks))
    t_quant = time.perf_counter() - t0
    # the GEMM rows need W quantized whole; that is not timed again (the W
    # share above already stands for it at the sampled rate)
    with ThreadPoolExecutor(cores) as ex:
        wparts = list(ex.map(lambda i: oracle.quantize(wb[i:i + 128], oracle.BLOCK_128x128),
                             range(0, N, 128)))
    ow = np.concatenate([c for c, _ in wparts])
    osw = np.concatenate([s for _, s in wparts])
    t1 = time.perf_counter()
    with ThreadPoolExecutor(cores) as ex:
        def rows_of(i):
            codes, scales = xres[i]
            n = codes.shape[0]
            return oracle.gemm_rows(codes, scales, oracle.BLOCK_1x128, ow, osw,
                                    oracle.BLOCK_128x128, np.arange(n))
        list(ex.map(rows_of, range(len(xres))))
    t_gemm = time.perf_counter() - t1
    # the sampled share of one step: rows/M of the GEMM and of X, wrows/N of W
    t_step = t_gemm + t_quant
    flops = 2.0 * rows * N * K
    return {
        "value": flops / t_step / 1e12,
        "unit": "TFLOP/s",
        "cores": cores,
        "kind": "oracle",
        "sample": "%d of %d rows of Y = X W^T (exact int64/binary128 oracle GEMM), "
                  "those rows of X quantized 1x128 and %d of %d rows of W quantized "
                  "128x128; %.1f s wall (%.1f s quantize, %.1f s GEMM)"
                  % (rows, M, wrows, N, t_step, t_quant, t_gemm),
    }


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
    }
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
