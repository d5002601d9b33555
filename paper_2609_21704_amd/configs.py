"""The five synthetic workloads: Qwen2.5-shaped weight-streaming stacks.

Every matrix is stored [n][k] (n outputs, k inputs).  A decoder layer streams
four weight matrices per token: the fused q|k|v projection, the output
projection o, the fused gate|up projection and the down projection; the
LM head closes the stack.  Fusing q|k|v and gate|up (rows concatenated) leaves
the bytes and the per-row quantization unchanged and mirrors the inputs they
share.  Weights are N(0, 0.02) fp16 (standard deviation 0.02), activations
N(0, 1) fp16, every tensor drawn from the config seed.
"""
from __future__ import annotations

from dataclasses import dataclass, field

HEAD_DIM = 128


@dataclass(frozen=True)
class Config:
    index: int
    name: str
    layers: int
    hidden: int
    intermediate: int
    q_heads: int
    kv_heads: int
    vocab: int
    draft_variant: str          # "int4" or "fp8"
    k: int                      # drafted tokens per round
    batch: int                  # sequences per round
    seed: int
    lm_head: bool = True        # False: synthetic draft logits ~ N(0, 2) instead of an LM head
    extra_variants: tuple = field(default=())

    @property
    def q_dim(self) -> int:
        return self.q_heads * HEAD_DIM

    @property
    def kv_dim(self) -> int:
        return self.kv_heads * HEAD_DIM

    def layer_matrices(self):
        """(name, n, k) of the four weight matrices of one decoder layer."""
        h = self.hidden
        return [
            ("qkv", self.q_dim + 2 * self.kv_dim, h),
            ("o", h, self.q_dim),
            ("gate_up", 2 * self.intermediate, h),
            ("down", h, self.intermediate),
        ]

    def matrices(self):
        mats = [(l, name, n, k) for l in range(self.layers) for name, n, k in self.layer_matrices()]
        if self.lm_head:
            mats.append((self.layers, "lm_head", self.vocab, self.hidden))
        return mats

    @property
    def draft_m(self) -> int:
        return self.batch

    @property
    def verify_m(self) -> int:
        return self.batch * (self.k + 1)

    def params(self) -> int:
        return sum(n * k for _, _, n, k in self.matrices())

    def bytes_per_weight(self, variant: str) -> float:
        return {"int4": 17.0 / 32.0, "fp8": 1.0, "f16": 2.0}[variant]

    def pass_bytes(self, variant: str) -> float:
        """Algorithmic weight bytes of one pass over the stack (FP8 adds 4 B per row)."""
        tot = 0.0
        for _, _, n, k in self.matrices():
            tot += n * k * self.bytes_per_weight(variant)
            if variant == "fp8":
                tot += 4 * n
        return tot

    def round_bytes(self) -> float:
        """k draft passes with the draft copy plus one verify pass with the FP16 parent."""
        return self.k * self.pass_bytes(self.draft_variant) + self.pass_bytes("f16")

    def describe(self) -> str:
        return (f"{self.name}: {self.layers} layers, hidden {self.hidden}, intermediate {self.intermediate}, "
                f"{self.q_heads} q / {self.kv_heads} kv heads of dim {HEAD_DIM}, "
                + (f"LM head {self.vocab}x{self.hidden}, " if self.lm_head else f"synthetic logits over {self.vocab}, ")
                + f"FP16 parent + {self.draft_variant.upper()} draft, k={self.k}, batch {self.batch}, "
                f"draft M={self.draft_m}, verify M={self.verify_m}, seed {self.seed}")


CONFIGS = [
    Config(0, "Qwen2.5-0.5B-shaped single layer", 1, 896, 4864, 7, 1, 4096, "int4", 4, 1, 0, lm_head=False,
           extra_variants=("fp8",)),
    Config(1, "Qwen2.5-1.5B-shaped stack", 28, 1536, 8960, 12, 2, 151936, "int4", 4, 1, 1, extra_variants=("fp8",)),
    Config(2, "Qwen2.5-7B-shaped stack", 28, 3584, 18944, 28, 4, 151936, "int4", 4, 1, 2),
    Config(3, "Qwen2.5-7B-shaped stack, batch 4", 28, 3584, 18944, 28, 4, 151936, "fp8", 8, 4, 3),
    Config(4, "Qwen2.5-32B-shaped stack", 64, 5120, 27648, 40, 8, 152064, "int4", 6, 1, 4),
]

HEADLINE = 2
