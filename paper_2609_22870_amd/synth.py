"""Seeded synthetic operands for the FP8 linear layer.

This module only draws random numbers and fixes the workload shapes; it
holds none of the method's arithmetic.  Both the oracle side and the HIP
side of every test and of the benchmark take their inputs from here, as the
same bf16 bytes.

The paper trains Qwen3-8B-Base, Qwen3-14B-Base and Qwen2.5-32B on math
datasets (Sec. 3 and Sec. 5.1-5.2) and benchmarks training throughput at 8B,
14B and 32B with 4K/8K/16K-token sequences (Sec. 5.3).  Neither weights nor
data are available, so the operands are seeded normal draws at the layer
shapes of those models:

* activations X ~ N(0, 1), with 1% of the input channels (columns along the
  contraction dimension) multiplied by 50 in fp32 before the single bf16
  rounding, as outlier channels;
* weights W ~ N(0, 0.02), stored [N, K] (output channel major);
* output gradients dY ~ N(0, 1e-3).

M = 16384 tokens is one 16K-context sequence; M = 256 is one decode step over
256 sequences.

For Calibrated Clipping (Sec. 4, Alg. 1) the inputs are per-token arrays of
one GRPO training batch (Appendix setup: 256 prompts, 8 responses each, 16K
context); see rl_batch.
"""
import torch

# (M, K, N) of the GEMM C[M, N] = A[M, K] B[N, K]^T, per named workload.
WORKLOADS = {
    "tiny_tensorwise": dict(shapes=[(128, 256, 256)], scaling="tensor"),
    "8b_ffn_up_fwd_blockwise": dict(shapes=[(16384, 4096, 12288)],
                                    scaling="block"),
    "8b_rowwise": dict(shapes=[(16384, 4096, 12288), (16384, 12288, 4096),
                               (16384, 4096, 6144)], scaling="row"),
    "8b_decode_blockwise": dict(shapes=[(256, 4096, 12288), (256, 12288, 4096)],
                                scaling="block"),
    # 32B-class MLP: hidden 5120, FFN 25600, one 16K-token sequence.
    # Listed as the GEMMs of the up and down projections in forward, dgrad
    # and wgrad layouts; "pass" names which.
    "32b_train_blockwise": dict(shapes=[(16384, 5120, 25600), (16384, 25600, 5120),
                                        (5120, 16384, 25600), (16384, 25600, 5120),
                                        (16384, 5120, 25600), (25600, 16384, 5120)],
                                passes=["fwd", "dgrad", "wgrad",
                                        "fwd", "dgrad", "wgrad"],
                                scaling="block"),
}

SIGMA_X, SIGMA_W, SIGMA_DY = 1.0, 0.02, 1e-3
OUTLIER_FRACTION, OUTLIER_GAIN = 0.01, 50.0


def seed_for(workload_index, role, shape_index=0):
    """Seed of one operand: 1000 * workload + 100 * shape + role, with roles
    X=0, W=1, dY=2, outlier-channel choice=3."""
    return 1000 * workload_index + 100 * shape_index + role


def normal_bf16(shape, sigma, seed, device="cpu", outlier_cols=None,
                gain=OUTLIER_GAIN):
    """N(0, sigma) drawn in fp32 from a seeded generator, optionally with the
    listed columns multiplied by `gain`, then rounded once to bf16."""
    gen = torch.Generator(device=device)
    gen.manual_seed(seed)
    x = torch.randn(shape, generator=gen, device=device, dtype=torch.float32)
    x.mul_(sigma)
    if outlier_cols is not None and len(outlier_cols):
        idx = torch.as_tensor(outlier_cols, device=device, dtype=torch.long)
        x[:, idx] *= gain
    return x.to(torch.bfloat16)


def outlier_columns(ncols, seed, fraction=OUTLIER_FRACTION):
    """round(fraction * ncols) distinct column indices drawn from a seed."""
    count = int(round(fraction * ncols))
    gen = torch.Generator()
    gen.manual_seed(seed)
    return torch.randperm(ncols, generator=gen)[:count].sort().values.tolist()


def activations(M, K, seed, outlier_seed, device="cpu"):
    return normal_bf16((M, K), SIGMA_X, seed, device,
                       outlier_cols=outlier_columns(K, outlier_seed))


def weights(N, K, seed, device="cpu"):
    return normal_bf16((N, K), SIGMA_W, seed, device)


def grads(M, N, seed, device="cpu"):
    return normal_bf16((M, N), SIGMA_DY, seed, device)


def weights_block_gains(N, K, seed, gain_seed, device="cpu"):
    """weights() with each 128 x 128 block (of rows and columns) multiplied
    by its own power of two 2^g, g drawn uniformly from -6 .. 6 with a
    seeded generator: exact in bf16, and the blocks' scales then differ by
    up to 2^12 instead of a few percent."""
    w = weights(N, K, seed, device)
    gen = torch.Generator()
    gen.manual_seed(gain_seed)
    g = torch.randint(-6, 7, ((N + 127) // 128, (K + 127) // 128), generator=gen)
    gains = torch.pow(2.0, g.to(torch.float32))
    gains = gains.repeat_interleave(128, 0)[:N].repeat_interleave(128, 1)[:, :K]
    return (w.to(torch.float32) * gains.to(w.device)).to(torch.bfloat16)


def bf16_bits(t):
    """bf16 tensor -> numpy uint16 bit patterns (CPU copy)."""
    return t.detach().cpu().contiguous().view(torch.int16).numpy().view("uint16")


# GRPO batch of the paper's 8B setup: prompts x responses per prompt, with
# response lengths drawn uniformly from [RL_MIN_LEN, RL_MAX_LEN] tokens.
RL_BATCH = dict(prompts=256, group=8)
RL_MIN_LEN, RL_MAX_LEN = 512, 8192


def rl_batch(prompts, group, seed, min_len=RL_MIN_LEN, max_len=RL_MAX_LEN, zero_adv=0.1,
             ratio_sigma=0.05, fp8_sigma=0.03, tis_sigma=0.02, tis_cap=2.0, device="cpu"):
    """Per-token float32 inputs of Calibrated Clipping for one batch, as a
    dict of 1-D tensors (adv, w_tis, pi_sampler, r_bf16, r_fp8), responses
    laid out one after another.  Stand-ins drawn from a seeded generator:

    * each response has one advantage for all its tokens, N(0, 1), or 0 for
      a fraction `zero_adv` of the responses (groups whose rewards all agree);
    * sampler token probabilities 1 / (1 + exp(-z)), z ~ N(3, 2);
    * BF16 importance ratios exp(N(0, ratio_sigma)); FP8 ratios are the BF16
      ones times exp(N(0, fp8_sigma)), the quantization noise;
    * TIS weights min(exp(N(0, tis_sigma)), tis_cap).
    """
    g = torch.Generator().manual_seed(seed)
    n_resp = prompts * group
    lens = torch.randint(min_len, max_len + 1, (n_resp,), generator=g)
    adv_resp = torch.randn(n_resp, generator=g)
    adv_resp[torch.rand(n_resp, generator=g) < zero_adv] = 0.0
    adv = torch.repeat_interleave(adv_resp, lens)
    n = adv.numel()
    pi = torch.sigmoid(3.0 + 2.0 * torch.randn(n, generator=g))
    r_bf16 = torch.exp(ratio_sigma * torch.randn(n, generator=g))
    r_fp8 = r_bf16 * torch.exp(fp8_sigma * torch.randn(n, generator=g))
    w = torch.clamp(torch.exp(tis_sigma * torch.randn(n, generator=g)), max=tis_cap)
    out = dict(adv=adv, w_tis=w, pi_sampler=pi, r_bf16=r_bf16, r_fp8=r_fp8)
    return {k: v.to(torch.float32).contiguous().to(device) for k, v in out.items()}
