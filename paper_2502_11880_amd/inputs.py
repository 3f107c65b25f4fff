"""Seeded synthetic inputs and workload shapes.

This module draws random numbers only: it holds none of the method's arithmetic (no ternarisation, no
quantisation, no packing), so the HIP path and the CPU oracle can both be fed from it.

Recipe (the paper's models are trained ternary LLMs whose shapes it does not list; these stand in for them):

* weights: fp32 N(0, 0.02), one generator per tensor (integer weights of C values: uniform over the set, or for
  C = 3 the frequencies of absmean-ternarised Gaussian weights);
* activations: fp32 N(0, 1), then exactly round(0.001 * M * K) distinct positions, drawn without
  replacement from the same generator, are multiplied by 20 (sign kept);
* seed of tensor i of workload c: 0xB17E7 + 1000 * c + i.
"""
from __future__ import annotations

import torch

SEED_BASE = 0xB17E7
OUTLIER_FRACTION = 0.001
OUTLIER_GAIN = 20.0
WEIGHT_STD = 0.02


def seed_for(workload: int, tensor_index: int) -> int:
    return SEED_BASE + 1000 * workload + tensor_index


def _generator(seed: int, device) -> torch.Generator:
    dev = torch.device(device)
    g = torch.Generator(device=dev)
    g.manual_seed(seed)
    return g


def weight_f32(N: int, K: int, seed: int, device="cpu") -> torch.Tensor:
    """fp32 [N, K] weights drawn from N(0, 0.02)."""
    g = _generator(seed, device)
    w = torch.empty((N, K), dtype=torch.float32, device=device)
    w.normal_(0.0, WEIGHT_STD, generator=g)
    return w


def int_weights(N: int, K: int, C: int, seed: int, device="cpu") -> torch.Tensor:
    """int8 [N, K] weights from the set of C consecutive integers -(C // 2) .. C - 1 - C // 2: for C = 3 with the
    frequencies of absmean-ternarised Gaussian weights (0 with probability 0.31), otherwise uniform."""
    g = _generator(seed, device)
    lo = -(C // 2)
    if C == 3:
        u = torch.rand((N, K), generator=g, device=device)
        w = torch.where(u < 0.345, -1, torch.where(u < 0.655, 0, 1))
    else:
        w = torch.randint(0, C, (N, K), generator=g, device=device) + lo
    return w.to(torch.int8)


def activation_f32(M: int, K: int, seed: int, device="cpu") -> torch.Tensor:
    """fp32 [M, K] activations drawn from N(0, 1) with 0.1% of the entries scaled by 20."""
    g = _generator(seed, device)
    x = torch.empty((M, K), dtype=torch.float32, device=device)
    x.normal_(0.0, 1.0, generator=g)
    n_out = int(round(OUTLIER_FRACTION * M * K))
    if n_out:
        pos = torch.randperm(M * K, generator=g, device=device)[:n_out]
        flat = x.view(-1)
        flat[pos] = flat[pos] * OUTLIER_GAIN
    return x


# Linear layers of each workload as (name, K, N, count).  Decode token counts and prefill token counts
# are listed per workload.
WORKLOADS = {
    0: dict(name="single-linear-1536x4096", linears=[("proj", 1536, 4096, 1)], tokens=[1]),
    1: dict(name="bitnet-3B-layer-decode",
            linears=[("q", 3200, 3200, 1), ("k", 3200, 3200, 1), ("v", 3200, 3200, 1), ("o", 3200, 3200, 1),
                     ("gate", 3200, 8640, 1), ("up", 3200, 8640, 1), ("down", 8640, 3200, 1)],
            tokens=[1]),
    2: dict(name="llama3-8B-1.58-layer-decode",
            linears=[("q", 4096, 4096, 1), ("k", 4096, 1024, 1), ("v", 4096, 1024, 1), ("o", 4096, 4096, 1),
                     ("gate", 4096, 14336, 1), ("up", 4096, 14336, 1), ("down", 14336, 4096, 1)],
            tokens=[1, 8]),
    3: dict(name="llama3-8B-1.58-layer-prefill",
            linears=[("q", 4096, 4096, 1), ("k", 4096, 1024, 1), ("v", 4096, 1024, 1), ("o", 4096, 4096, 1),
                     ("gate", 4096, 14336, 1), ("up", 4096, 14336, 1), ("down", 14336, 4096, 1)],
            tokens=[512, 2048]),
    4: dict(name="ternary-100B-stack-decode",
            linears=[("q", 12288, 12288, 1), ("k", 12288, 12288, 1), ("v", 12288, 12288, 1),
                     ("o", 12288, 12288, 1), ("gate", 12288, 33024, 1), ("up", 12288, 33024, 1),
                     ("down", 33024, 12288, 1)],
            tokens=[1], layers=56),
}

# Linears that read the same quantised activation row within one layer: (q, k, v), (o), (gate, up), (down).
ACTIVATION_GROUPS = [("q", "k", "v"), ("o",), ("gate", "up"), ("down",)]
