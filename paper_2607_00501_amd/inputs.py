"""Seeded synthetic inputs (weights N(0, 0.02^2), activations and router
logits N(0, 1)), shared by the GPU path and the CPU oracle.

This module holds no arithmetic of the method: it only draws numbers.  Host
arrays come from numpy's PCG64 generator; large device tensors come from a
seeded torch CUDA generator (the same seed always yields the same bytes on
the same software stack).  Whichever side consumes an input, both sides are
handed the very same bytes.
"""

from __future__ import annotations

import numpy as np

WEIGHT_SIGMA = 0.02

# tensor ids inside a seed (q, k, v, o, gate, up, down, lm_head, x, logits)
TENSOR_ID = {"q": 0, "k": 1, "v": 2, "o": 3, "gate": 4, "up": 5, "down": 6, "lm_head": 7, "x": 8,
             "logits": 9, "emb": 10, "attn_norm": 11, "ffn_norm": 12, "norm": 13, "cache": 14}


def seed_for(config: int, layer: int, tensor: str, call: int = 0) -> int:
    """Seed of one tensor of a workload: config, layer (or expert) and tensor
    name; `call` separates repeated activations of the same projection."""
    return 1_000_003 * config + 1009 * layer + 17 * TENSOR_ID[tensor] + 7_919_993 * call


def weights_np(seed: int, shape, sigma: float = WEIGHT_SIGMA) -> np.ndarray:
    """fp32 weights ~ N(0, sigma^2)."""
    rng = np.random.default_rng(seed)
    return rng.standard_normal(shape, dtype=np.float32) * np.float32(sigma)


def activations_np(seed: int, shape) -> np.ndarray:
    """fp16 activations ~ N(0, 1) (drawn in fp32, rounded to fp16)."""
    rng = np.random.default_rng(seed)
    return rng.standard_normal(shape, dtype=np.float32).astype(np.float16)


def norm_weights_np(seed: int, shape) -> np.ndarray:
    """fp16 norm gains ~ 1 + N(0, 0.1^2) (drawn in fp32, rounded to fp16)."""
    rng = np.random.default_rng(seed)
    return (1.0 + 0.1 * rng.standard_normal(shape, dtype=np.float32)).astype(np.float16)


def logits_np(seed: int, shape) -> np.ndarray:
    """fp32 router logits ~ N(0, 1)."""
    rng = np.random.default_rng(seed)
    return rng.standard_normal(shape, dtype=np.float32)


def _torch_gen(seed: int, device):
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return g


def weights_dev(seed: int, shape, device="cuda", sigma: float = WEIGHT_SIGMA):
    """fp32 weights ~ N(0, sigma^2) drawn on the device (for large tensors)."""
    import torch
    w = torch.randn(shape, generator=_torch_gen(seed, device), device=device, dtype=torch.float32)
    return w.mul_(sigma)


def activations_dev(seed: int, shape, device="cuda"):
    import torch
    return torch.randn(shape, generator=_torch_gen(seed, device), device=device,
                       dtype=torch.float32).to(torch.float16)


def logits_dev(seed: int, shape, device="cuda"):
    import torch
    return torch.randn(shape, generator=_torch_gen(seed, device), device=device, dtype=torch.float32)
