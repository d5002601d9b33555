"""Seeded synthetic inputs for the SpecQuant hot path.

This module holds no SpecQuant arithmetic: it only draws random tensors with
the shapes and value laws of the workloads (weights ~ N(0, 0.02) in fp16,
activations ~ N(0, 1) in fp16, logits ~ N(0, sigma) in fp32, 24-bit uniforms).
Both the GPU path and the CPU oracle consume its tensors; the oracle always
receives the exact bytes the GPU received.  N(mu, sigma) names the standard
deviation sigma.
"""
from __future__ import annotations

import torch


def _gen(seed: int, device) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(int(seed) & 0x7FFFFFFFFFFFFFFF)
    return g


def stream_seed(seed: int, *ids: int) -> int:
    """Derive a sub-seed for one tensor from a config seed and integer ids."""
    h = (int(seed) * 0x9E3779B97F4A7C15) & 0xFFFFFFFFFFFFFFFF
    for i in ids:
        h ^= (int(i) + 0x632BE59BD9B4E019 + ((h << 6) & 0xFFFFFFFFFFFFFFFF) + (h >> 2)) & 0xFFFFFFFFFFFFFFFF
        h = (h * 0xBF58476D1CE4E5B9) & 0xFFFFFFFFFFFFFFFF
    return h & 0x7FFFFFFFFFFFFFFF


def normal_f16(shape, std: float, seed: int, device="cpu") -> torch.Tensor:
    """fp16 tensor with N(0, std) entries (drawn in fp32, rounded once to fp16)."""
    g = _gen(seed, device)
    t = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
    t.mul_(std)
    return t.to(torch.float16)


def normal_f32(shape, std: float, seed: int, device="cpu") -> torch.Tensor:
    g = _gen(seed, device)
    t = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
    return t.mul_(std)


def uniform_u24(shape, seed: int, device="cpu") -> torch.Tensor:
    """Integers uniform in [0, 2^24) stored as int32 (the u24 uniforms)."""
    g = _gen(seed, device)
    return torch.randint(0, 1 << 24, shape, generator=g, device=device, dtype=torch.int64).to(torch.int32)


def tokens(shape, vocab: int, seed: int, device="cpu") -> torch.Tensor:
    g = _gen(seed, device)
    return torch.randint(0, vocab, shape, generator=g, device=device, dtype=torch.int64).to(torch.int32)
