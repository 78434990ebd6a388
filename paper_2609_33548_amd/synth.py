"""Seeded synthetic inputs shared by the tests, the smoke check and the bench.

This module draws inputs only (latent weights, activations, targets, token
ids); it holds none of the TerMeZO arithmetic.  Host-side draws use numpy's
PCG64 generator; large device-side draws use torch's generator on the device.

Distributions (stand-ins for the paper's pretrained models and datasets, which
are not available): latent weights N(0, 0.02^2), activations and regression
targets N(0, 1), token ids uniform over the vocabulary.
"""
from __future__ import annotations

import numpy as np

LATENT_STD = 0.02


def to_bf16_values(x: np.ndarray) -> np.ndarray:
    """Round finite fp32 values to the nearest bfloat16 (ties to even), kept as fp32.
    (In 32-bit unsigned arithmetic: a finite value's bits plus 0x8000 stay below 2^32.)"""
    b = np.array(x, dtype=np.float32, copy=True, order="C").view(np.uint32)
    lsb = (b >> np.uint32(16)) & np.uint32(1)
    b += np.uint32(0x7FFF)
    b += lsb
    b &= np.uint32(0xFFFF0000)
    return b.view(np.float32)


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """Upper 16 bits of fp32 values that are already bfloat16 values."""
    return (np.ascontiguousarray(x, np.float32).view(np.uint32) >> 16).astype(np.uint16)


def latents(seed: int, sizes, bf16: bool = False) -> np.ndarray:
    """All latent weights, concatenated in layer order, as fp32 (bf16 values if bf16)."""
    rng = np.random.default_rng(seed)
    w = (rng.standard_normal(int(sum(sizes)), dtype=np.float32) * np.float32(LATENT_STD))
    w = w.astype(np.float32)
    return to_bf16_values(w) if bf16 else w


def activations(seed: int, M: int, K: int, bf16: bool = False) -> np.ndarray:
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((M, K), dtype=np.float32)
    return to_bf16_values(x) if bf16 else x


def tokens(seed: int, B: int, S: int, vocab: int) -> np.ndarray:
    rng = np.random.default_rng(seed)
    return rng.integers(0, vocab, size=(B, S), dtype=np.int32)


def torch_latents(seed: int, n: int, dtype, device):
    """Device-side draw for full-size workloads (torch generator on the device)."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    w = torch.empty(n, dtype=torch.float32, device=device)
    chunk = 1 << 28
    for s in range(0, n, chunk):
        e = min(n, s + chunk)
        w[s:e].normal_(0.0, LATENT_STD, generator=g)
    return w.to(dtype)


def torch_normal(seed: int, shape, dtype, device):
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return torch.randn(shape, generator=g, dtype=torch.float32, device=device).to(dtype)


def torch_tokens(seed: int, B: int, S: int, vocab: int, device):
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return torch.randint(0, vocab, (B, S), generator=g, dtype=torch.int32, device=device)
