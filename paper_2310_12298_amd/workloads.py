"""Seeded synthetic workloads for the Jorge step: layer shapes and inputs.

This module holds no arithmetic of the method: only layer-shape lists and the
seeded generators of gradients and initial parameters that the GPU path, the
tests and the benchmark all draw their inputs from.

Gradients are fresh every step: G[layer, t] is drawn from
numpy.random.default_rng([seed, layer, t]) as float32 N(0, sigma^2).
Initial parameters use the same generator with t = 2**31 - 1, scaled by
sqrt(2 / n) (He initialisation of an m x n weight).
"""
from __future__ import annotations

import numpy as np

THETA_STREAM = 2 ** 31 - 1


def resnet50_weight_shapes() -> list[tuple[int, int]]:
    """The 53 convolution weights and the fc weight of torchvision ResNet-50 (v1.5).

    Each N-d weight is collapsed to out x (in * kh * kw), the 2-D view the
    paper optimises (Section 3).
    """
    shapes = [(64, 3 * 7 * 7)]                           # stem 7x7, 3 -> 64
    in_ch = 64
    for width, blocks in ((64, 3), (128, 4), (256, 6), (512, 3)):
        out_ch = 4 * width
        for b in range(blocks):
            shapes.append((width, in_ch))                # 1x1 reduce
            shapes.append((width, width * 9))            # 3x3
            shapes.append((out_ch, width))               # 1x1 expand
            if b == 0:
                shapes.append((out_ch, in_ch))           # 1x1 downsample
            in_ch = out_ch
    shapes.append((1000, 2048))                          # fc
    return shapes


def many_small_shapes(num_layers: int = 512, seed: int = 0) -> list[tuple[int, int]]:
    """512 layers with m, n drawn uniformly from {32, 64, 128, 256}."""
    dims = np.random.default_rng(seed).choice([32, 64, 128, 256], size=(num_layers, 2))
    return [(int(a), int(b)) for a, b in dims]


# name -> (shapes, gradient sigma, steps of the full run)
CONFIGS = {
    "single_64x576": ([(64, 576)], 1e-2, 10),
    "single_512x4608": ([(512, 4608)], 1e-3, 100),
    "resnet50": (resnet50_weight_shapes(), 1e-3, 50),
    "large_dense": ([(4096, 4096)] * 8 + [(4096, 1024)] * 8, 1e-3, 20),
    "many_small": (many_small_shapes(), 1e-2, 200),
}

# Hyperparameters shared by the synthetic workloads.
DEFAULT_HPARAMS = dict(lr=0.1, beta2=0.9, beta1=0.9, weight_decay=5e-5, eps=1e-6,
                       precond_interval=1)


def gradient(seed: int, layer: int, t: int, shape, sigma: float) -> np.ndarray:
    """G[layer, t]: float32 row-major m x n, iid N(0, sigma^2)."""
    rng = np.random.default_rng([seed, layer, t])
    return rng.standard_normal(tuple(shape), dtype=np.float32) * np.float32(sigma)


def initial_params(seed: int, layer: int, shape) -> np.ndarray:
    """theta_0[layer]: float32 m x n, N(0, 2/n)."""
    rng = np.random.default_rng([seed, layer, THETA_STREAM])
    m, n = shape
    return rng.standard_normal((m, n), dtype=np.float32) * np.float32(np.sqrt(2.0 / n))


def param_count(shapes) -> int:
    return int(sum(m * n for m, n in shapes))


def _stream_seed(seed: int, layer: int, t: int) -> int:
    """64-bit seed of the (seed, layer, t) stream, from numpy's SeedSequence."""
    return int(np.random.SeedSequence([seed, layer, t]).generate_state(1, np.uint64)[0] >> 1)


def device_gradient(seed: int, layer: int, t: int, shape, sigma: float, device: str = "cuda"):
    """G[layer, t] drawn on the device (torch's Philox generator), N(0, sigma^2) fp32.

    A different stream from gradient(): used where host generation would take
    longer than the measurement (pre-staging many full-size gradient sets).
    """
    import torch
    gen = torch.Generator(device=device)
    gen.manual_seed(_stream_seed(seed, layer, t))
    return torch.randn(tuple(shape), generator=gen, device=device, dtype=torch.float32).mul_(sigma)


def device_initial_params(seed: int, layer: int, shape, device: str = "cuda"):
    """theta_0[layer] drawn on the device: N(0, 2/n) fp32."""
    m, n = shape
    return device_gradient(seed, layer, THETA_STREAM, shape, float(np.sqrt(2.0 / n)), device)
