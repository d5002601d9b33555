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


# ------------------------------------------------------------ prompt texts
# Words of the synthetic prompt grammar (invented names and plain vocabulary).
_NOUNS = ("river", "engine", "market", "garden", "signal", "ledger", "bridge", "harvest", "circuit", "library",
          "orbit", "painting", "contract", "forest", "protein", "budget", "voyage", "lantern", "theory", "village")
_VERBS = ("explain", "compare", "describe", "estimate", "summarise", "predict", "measure", "design", "justify",
          "translate")
_ADJS = ("ancient", "rapid", "fragile", "distant", "efficient", "hidden", "modest", "curious", "stable", "narrow")
_NAMES = ("Varenholt", "Quillon", "Maribeth Oduya", "Port Celestine", "the Haldane Institute", "Tovrik", "NORDAX",
          "Elsbeth Crane", "Lake Imari", "the Corvanne Group", "Dr. Pell", "Ashgrove")
_SUBS = ("because", "although", "which", "while", "if", "that", "unless", "whereas", "since", "when")


def prompt_texts(n: int, seed: int) -> list[str]:
    """n seeded prompts with a mix of lengths and structures: short direct
    questions, instructions of a few sentences, and long multi-clause
    problems with numbers, names and parentheses."""
    import random
    rng = random.Random(stream_seed(seed, 0x7E47))
    out = []
    for _ in range(n):
        style = rng.random()
        if style < 0.3:
            sents = 1
            clause_p, entity_p, words = 0.05, 0.15, rng.randint(3, 9)
        elif style < 0.8:
            sents = rng.randint(1, 4)
            clause_p, entity_p, words = 0.2, 0.3, rng.randint(6, 16)
        else:
            sents = rng.randint(3, 12)
            clause_p, entity_p, words = 0.45, 0.5, rng.randint(10, 26)
        text = []
        for _ in range(sents):
            w = [rng.choice(_VERBS).capitalize(), "the", rng.choice(_ADJS), rng.choice(_NOUNS)]
            while len(w) < words:
                r = rng.random()
                if r < clause_p:
                    w += [",", rng.choice(_SUBS), "the", rng.choice(_NOUNS), rng.choice(("is", "was", "seems"))]
                elif r < clause_p + entity_p * 0.5:
                    w += ["of", rng.choice(_NAMES)]
                elif r < clause_p + entity_p * 0.7:
                    w += ["in", str(rng.randint(2, 2099))]
                elif r < clause_p + entity_p * 0.8:
                    w += ["(", "see", rng.choice(_NAMES), ")"]
                else:
                    w += [rng.choice(("and", "with", "for", "near")), rng.choice(_ADJS), rng.choice(_NOUNS)]
            text.append(" ".join(w).replace(" ,", ",").replace("( ", "(").replace(" )", ")") +
                        rng.choice((".", "?", ".")))
        out.append(" ".join(text))
    return out
