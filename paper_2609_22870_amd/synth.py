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


def bf16_bits(t):
    """bf16 tensor -> numpy uint16 bit patterns (CPU copy)."""
    return t.detach().cpu().contiguous().view(torch.int16).numpy().view("uint16")
