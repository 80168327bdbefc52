"""Seeded synthetic inputs for DKM clustering runs.

This module only draws numbers; it holds none of DKM's arithmetic.  The tests,
the smoke check and the benchmark all take their inputs from here, so the HIP
path and the CPU oracle see identical data.

Recipe (the paper's workload is LLaMA-7B weights fine-tuned in 16 bits; no
weights are available, so these draws stand in for them):

* weights: fp32 draws from N(0, 0.02^2) rounded to fp16, or for bf16 weights
  to bfloat16 (round-to-nearest-even either way);
  with ``outliers`` each element independently, with probability 1e-3, is
  replaced before rounding by a draw from N(0, 0.2^2);
* initial centroids: the k evenly spaced quantiles of the fp16 values, i.e. the
  sorted value at 0-based rank floor((j + 1/2) N / k), as fp32 (exact);
* upstream gradient dL/dW~: fp32 draws from N(0, 1).

Generators are numpy PCG64 streams; seeds follow 1000*config + matrix index for
weights and that plus 500 for gradients.  The 32-layer stack (6.5e9 weights) is
drawn on the GPU instead, from torch's device generator with the same seeds and
the same recipe (``*_device``); a test copies a sampled matrix back to the host.
"""
from __future__ import annotations

import numpy as np

SIGMA = 0.02
OUTLIER_SIGMA = 0.2
OUTLIER_P = 1e-3
TAU = 2e-3
ITERS = 5

# LLaMA-7B decoder-layer projection shapes (rows x cols).
LLAMA7B_LAYER = (
    ("q_proj", 4096, 4096),
    ("k_proj", 4096, 4096),
    ("v_proj", 4096, 4096),
    ("o_proj", 4096, 4096),
    ("gate_proj", 11008, 4096),
    ("up_proj", 11008, 4096),
    ("down_proj", 4096, 11008),
)

# The five workloads: name -> (matrices as (name, rows, cols), bits list, outliers).
WORKLOADS = {
    1: dict(name="single_256x256", mats=(("w", 256, 256),), bits=(3,), outliers=False),
    2: dict(name="attn_proj_4096x4096", mats=(("w", 4096, 4096),), bits=(3,), outliers=False),
    3: dict(name="mlp_11008x4096_outliers", mats=(("w", 11008, 4096),), bits=(3, 4), outliers=True),
    4: dict(name="llama7b_decoder_layer", mats=LLAMA7B_LAYER, bits=(3,), outliers=False),
    5: dict(name="llama7b_32_layer_stack",
            mats=tuple(("L%d.%s" % (l, m), r, c) for l in range(32) for (m, r, c) in LLAMA7B_LAYER),
            bits=(3, 2, 4), outliers=False),
}


def weight_seed(config: int, matrix: int) -> int:
    return 1000 * config + matrix


def grad_seed(config: int, matrix: int) -> int:
    return 1000 * config + matrix + 500


def fp16_weights(n: int, seed: int, outliers: bool = False) -> np.ndarray:
    """n fp16 weights as raw bit patterns (uint16)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    w = rng.standard_normal(n, dtype=np.float32)
    w *= np.float32(SIGMA)
    if outliers:
        mask = rng.random(n, dtype=np.float32) < np.float32(OUTLIER_P)
        m = int(mask.sum())
        w[mask] = rng.standard_normal(m, dtype=np.float32) * np.float32(OUTLIER_SIGMA)
    return w.astype(np.float16).view(np.uint16)


def bf16_weights(n: int, seed: int, outliers: bool = False) -> np.ndarray:
    """The same fp32 draws as fp16_weights, rounded to bfloat16 (to nearest,
    ties to even) instead: n bf16 weights as raw bit patterns (uint16)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    w = rng.standard_normal(n, dtype=np.float32)
    w *= np.float32(SIGMA)
    if outliers:
        mask = rng.random(n, dtype=np.float32) < np.float32(OUTLIER_P)
        m = int(mask.sum())
        w[mask] = rng.standard_normal(m, dtype=np.float32) * np.float32(OUTLIER_SIGMA)
    u = w.view(np.uint32).astype(np.uint64)
    return ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)


def weights(n: int, seed: int, outliers: bool = False, fmt: str = "fp16") -> np.ndarray:
    """fp16_weights or bf16_weights by format name."""
    return (bf16_weights if fmt == "bf16" else fp16_weights)(n, seed, outliers)


def values(keys: np.ndarray, fmt: str = "fp16") -> np.ndarray:
    """16-bit patterns -> their fp32 values (exact)."""
    u = np.asarray(keys, dtype=np.uint16).ravel()
    if fmt == "bf16":
        return (u.astype(np.uint32) << 16).view(np.float32)
    return u.view(np.float16).astype(np.float32)


def quantile_init(keys: np.ndarray, k: int, fmt: str = "fp16") -> np.ndarray:
    """The k evenly spaced quantiles of the weight values (fp32, exact)."""
    vals = values(keys, fmt)
    n = vals.size
    ranks = np.array([((2 * j + 1) * n) // (2 * k) for j in range(k)], dtype=np.int64)
    part = np.partition(vals, np.unique(ranks))
    return part[ranks].astype(np.float32)


def two_cluster_weights(n_bulk: int, n_far: int, far_mean: float, far_sigma: float, seed: int,
                        bulk_sigma: float = 0.01) -> np.ndarray:
    """n_bulk fp32 draws from N(0, bulk_sigma^2) followed by n_far draws from
    N(far_mean, far_sigma^2), rounded to fp16 (raw bit patterns, uint16).  A
    small far group next to a bulk lets a centroid be empty in one iteration
    and occupied in the next."""
    rng = np.random.Generator(np.random.PCG64(seed))
    w = np.concatenate([rng.standard_normal(n_bulk) * bulk_sigma,
                        far_mean + rng.standard_normal(n_far) * far_sigma])
    return w.astype(np.float32).astype(np.float16).view(np.uint16)


def upstream_grad(n: int, seed: int) -> np.ndarray:
    """dL/dW~ ~ N(0, 1), fp32."""
    rng = np.random.Generator(np.random.PCG64(seed))
    return rng.standard_normal(n, dtype=np.float32)


def fp16_weights_device(n: int, seed: int, device, outliers: bool = False, fmt: str = "fp16"):
    """n fp16 (or, with fmt="bf16", bf16) weights as raw bit patterns
    (torch.int16 on ``device``), drawn by torch's generator on that device
    (same recipe as fp16_weights; torch rounds to nearest even)."""
    import torch
    gen = torch.Generator(device=device)
    gen.manual_seed(seed)
    w = torch.randn(n, generator=gen, device=device, dtype=torch.float32)
    w *= SIGMA
    if outliers:
        mask = torch.rand(n, generator=gen, device=device) < OUTLIER_P
        w[mask] = torch.randn(int(mask.sum()), generator=gen, device=device) * OUTLIER_SIGMA
    return w.to(torch.bfloat16 if fmt == "bf16" else torch.float16).view(torch.int16)


def quantile_init_device(keys, k: int, fmt: str = "fp16"):
    """quantile_init for device keys (torch.int16 bit patterns): fp32 on the same device."""
    import torch
    n = keys.numel()
    vals = torch.sort(keys.view(torch.bfloat16 if fmt == "bf16" else torch.float16).float()).values
    ranks = torch.tensor([((2 * j + 1) * n) // (2 * k) for j in range(k)], device=keys.device)
    return vals[ranks].contiguous()


def upstream_grad_device(n: int, seed: int, device):
    """dL/dW~ ~ N(0, 1), fp32, drawn on ``device``."""
    import torch
    gen = torch.Generator(device=device)
    gen.manual_seed(seed)
    return torch.randn(n, generator=gen, device=device, dtype=torch.float32)
