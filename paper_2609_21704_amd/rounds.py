"""One speculative round of SpecQuant on one GPU (SS III-D: draft generation,
parent verification, token acceptance or correction).

A round drafts k tokens per sequence with the quantized draft copy (k passes of
draft GEMVs at m = batch, each followed by a draft-token draw), verifies them
with the FP16 parent in one pass at m = batch * (k + 1), then accepts or
corrects.  Every step runs in the SpecQuant HIP kernels; torch only owns the
buffers and the stream.  The weight-streaming stack carries no attention or
normalisation, so each projection reads its own pre-drawn activation.

The parent's logits for the drafted positions are synthesised from the draft
logits: target row i = draft logits of step i + N(0, 0.5) noise (i < k); the
bonus row k is the parent LM head's output for the last verified position.
"""
from __future__ import annotations

from dataclasses import dataclass

import torch

from . import _lib as sq
from . import synth
from .configs import Config

# tensor ids for synth.stream_seed(config seed, kind, ...)
_W, _XD, _XV, _XLMD, _XLMV, _EPS, _UD, _UA, _DL, _BONUS, _XDIRECT = range(11)


class Stack:
    """Device-resident FP16 parent and its quantized draft copy."""

    def __init__(self, cfg: Config, device, variant: str | None = None, layers: int | None = None,
                 keep_f16: bool = True):
        self.cfg = cfg
        self.device = torch.device(device)
        self.variant = variant or cfg.draft_variant
        self.layers = cfg.layers if layers is None else layers
        self.w16 = {}      # (layer, name) -> fp16 [n][k]
        self.draft = {}    # (layer, name) -> (codes, scales[, zeros])
        mats = [(l, name, n, k) for (l, name, n, k) in cfg.matrices() if l < self.layers or name == "lm_head"]
        self.mats = mats
        for l, name, n, k in mats:
            mid = 1000 * (l + 1) + ["qkv", "o", "gate_up", "down", "lm_head"].index(name)
            w = synth.normal_f16((n, k), 0.02, synth.stream_seed(cfg.seed, _W, mid), self.device)
            if self.variant == "int4":
                self.draft[(l, name)] = sq.sq_quantize_int4_g128(w)
            elif self.variant == "fp8":
                self.draft[(l, name)] = sq.sq_quantize_fp8_e4m3(w)
            elif self.variant != "none":  # "none": the parent alone, no draft copy
                raise ValueError(f"unknown draft variant {self.variant!r}")
            if keep_f16:
                self.w16[(l, name)] = w
            else:
                del w

    def sibling(self, variant: str) -> "Stack":
        """The same FP16 parent with another quantized copy (every variant of
        SS III-A derives from the one parent): shares the FP16 matrices."""
        if not self.w16:
            raise ValueError("a sibling needs the FP16 matrices")
        if variant not in ("int4", "fp8"):
            raise ValueError(f"unknown draft variant {variant!r}")
        other = Stack.__new__(Stack)
        other.cfg, other.device, other.variant, other.layers, other.mats = (self.cfg, self.device, variant, self.layers,
                                                                             self.mats)
        other.w16 = self.w16
        other.draft = {key: (sq.sq_quantize_int4_g128(w) if variant == "int4" else sq.sq_quantize_fp8_e4m3(w))
                       for key, w in self.w16.items()}
        return other

    def draft_gemv(self, key, x, y):
        if self.variant == "int4":
            codes, scales, zeros = self.draft[key]
            sq.sq_qgemv_w4a16(x, codes, scales, zeros, y=y)
        else:
            codes, scales = self.draft[key]
            sq.sq_qgemv_w8a16(x, codes, scales, y=y)

    def verify_gemm(self, key, x, y):
        sq.sq_verify_gemm_f16(x, self.w16[key], y=y)

    # The decoder's fused forms (False: the shape's kernel has none, nothing enqueued).
    def draft_gemv_rmsnorm(self, key, h, norm_w, eps, group, y) -> bool:
        if self.variant != "int4":
            return False
        codes, scales, zeros = self.draft[key]
        return sq.sq_qgemv_w4a16_rmsnorm(h, norm_w, eps, codes, scales, zeros, group=group, y=y)

    def draft_gemv_rmsnorm_silu(self, key, h, norm_w, eps, t) -> bool:
        if self.variant != "int4":
            return False
        codes, scales, zeros = self.draft[key]
        return sq.sq_qgemv_w4a16_rmsnorm_silu(h, norm_w, eps, codes, scales, zeros, t)

    def verify_gemm_rmsnorm(self, key, h, norm_w, eps, group, y) -> bool:
        return sq.sq_verify_gemm_f16_rmsnorm(h, norm_w, eps, self.w16[key], group=group, y=y)

    def draft_gemv_acc(self, key, x, y) -> bool:
        if self.variant != "int4":
            return False
        codes, scales, zeros = self.draft[key]
        return sq.sq_qgemv_w4a16_acc(x, codes, scales, zeros, y)

    def verify_gemm_acc(self, key, x, y) -> bool:
        return sq.sq_verify_gemm_f16_acc(x, self.w16[key], y)


@dataclass
class RoundBuffers:
    xd: dict            # (step, layer, name) -> fp16 [B][k_in]
    xv: dict            # (layer, name) -> fp16 [B(k+1)][k_in]
    yd: dict            # name -> fp16 [B][n] (draft outputs, overwritten per layer)
    yv: dict            # name -> fp16 [B(k+1)][n]
    draft_logits: torch.Tensor    # f32 [k][B][V]
    target_logits: torch.Tensor   # f32 [B][k+1][V]
    eps: torch.Tensor             # f32 [B][k][V]
    draft_tokens: torch.Tensor    # i32 [k][B]
    u_draft: torch.Tensor         # i32 [k][B]   (current round)
    u_accept: torch.Tensor        # i32 [B][k+1] (current round)
    n_accepted: torch.Tensor      # i32 [B]
    next_token: torch.Tensor      # i32 [B]
    scratch_n: torch.Tensor       # i32 [B]


class Round:
    """Draft k tokens, verify, accept: the hot path of one SpecQuant round."""

    def __init__(self, stack: Stack, temperature: float = 1.0):
        self.stack = stack
        cfg = self.cfg = stack.cfg
        dev = stack.device
        self.temperature = float(temperature)
        B, k, V = cfg.batch, cfg.k, cfg.vocab
        seed = cfg.seed
        L = stack.layers
        xd, xv, yd, yv = {}, {}, {}, {}
        for name, n, kin in cfg.layer_matrices():
            yd[name] = torch.empty((B, n), dtype=torch.float16, device=dev)
            yv[name] = torch.empty((B * (k + 1), n), dtype=torch.float16, device=dev)
            for l in range(L):
                mid = 1000 * (l + 1) + ["qkv", "o", "gate_up", "down"].index(name)
                for i in range(k):
                    xd[(i, l, name)] = synth.normal_f16((B, kin), 1.0, synth.stream_seed(seed, _XD, mid, i), dev)
                xv[(l, name)] = synth.normal_f16((B * (k + 1), kin), 1.0, synth.stream_seed(seed, _XV, mid), dev)
        if cfg.lm_head:
            for i in range(k):
                xd[(i, L, "lm_head")] = synth.normal_f16((B, cfg.hidden), 1.0, synth.stream_seed(seed, _XLMD, i), dev)
            xv[(L, "lm_head")] = synth.normal_f16((B * (k + 1), cfg.hidden), 1.0,
                                                  synth.stream_seed(seed, _XLMV), dev)
            draft_logits = torch.empty((k, B, V), dtype=torch.float32, device=dev)
        else:
            draft_logits = synth.normal_f32((k, B, V), 2.0, synth.stream_seed(seed, _DL), dev)
        self.bonus = None if cfg.lm_head else synth.normal_f32((B, V), 2.0, synth.stream_seed(seed, _BONUS), dev)
        self.buf = RoundBuffers(
            xd=xd, xv=xv, yd=yd, yv=yv, draft_logits=draft_logits,
            target_logits=torch.empty((B, k + 1, V), dtype=torch.float32, device=dev),
            eps=synth.normal_f32((B, k, V), 0.5, synth.stream_seed(seed, _EPS), dev),
            draft_tokens=torch.zeros((k, B), dtype=torch.int32, device=dev),
            u_draft=torch.zeros((k, B), dtype=torch.int32, device=dev),
            u_accept=torch.zeros((B, k + 1), dtype=torch.int32, device=dev),
            n_accepted=torch.zeros((B,), dtype=torch.int32, device=dev),
            next_token=torch.zeros((B,), dtype=torch.int32, device=dev),
            scratch_n=torch.zeros((B,), dtype=torch.int32, device=dev),
        )
        self.graph = None

    # ------------------------------------------------------------ phases
    def draft_step(self, i: int, on_gemv=None):
        """Draft pass i: every layer's projections, the LM head, then the draw of token i."""
        st, b, cfg = self.stack, self.buf, self.cfg
        for l in range(st.layers):
            for name, _, _ in cfg.layer_matrices():
                if on_gemv:
                    on_gemv(True)
                st.draft_gemv((l, name), b.xd[(i, l, name)], b.yd[name])
                if on_gemv:
                    on_gemv(False)
        if cfg.lm_head:
            if on_gemv:
                on_gemv(True)
            st.draft_gemv((cfg.layers, "lm_head"), b.xd[(i, st.layers, "lm_head")], b.draft_logits[i])
            if on_gemv:
                on_gemv(False)
        # draw x_i ~ q_i: a plain sampler call (kd = 0) on draft row i
        B, V = cfg.batch, cfg.vocab
        sq.sq_spec_accept(None, b.draft_logits[i].view(B, 1, V), None, b.u_draft[i].view(B, 1),
                          self.temperature, n_accepted=b.scratch_n, next_token=b.draft_tokens[i])

    def verify(self):
        st, b, cfg = self.stack, self.buf, self.cfg
        for l in range(st.layers):
            for name, _, _ in cfg.layer_matrices():
                st.verify_gemm((l, name), b.xv[(l, name)], b.yv[name])
        k = cfg.k
        if cfg.lm_head:
            st.verify_gemm((cfg.layers, "lm_head"), b.xv[(st.layers, "lm_head")],
                           b.target_logits.view(cfg.batch * (k + 1), cfg.vocab))
        else:
            b.target_logits[:, k].copy_(self.bonus)
        # the parent's rows for the drafted positions: draft logits + N(0, 0.5)
        torch.add(b.draft_logits.permute(1, 0, 2), b.eps, out=b.target_logits[:, :k])

    def accept(self):
        b = self.buf
        sq.sq_spec_accept(b.draft_logits, b.target_logits, b.draft_tokens, b.u_accept, self.temperature,
                          n_accepted=b.n_accepted, next_token=b.next_token)

    def run(self, on_gemv=None):
        for i in range(self.cfg.k):
            self.draft_step(i, on_gemv)
        self.verify()
        self.accept()

    # ------------------------------------------------------------ graphs
    def capture(self):
        """Capture one round as a HIP graph (run once eagerly first so the
        library's workspace exists before capture)."""
        self.run()
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            self.run()
        torch.cuda.synchronize()
        self.graph = g
        return g

    def set_uniforms(self, u_draft: torch.Tensor, u_accept: torch.Tensor):
        self.buf.u_draft.copy_(u_draft)
        self.buf.u_accept.copy_(u_accept)

    def replay(self):
        self.graph.replay()


class DirectDecode:
    """Direct parent inference (SS III-D.5), the plain-decoding baseline the
    paper compares against: one token per sequence per step, every FP16
    matrix streamed once at m = batch rows (the verify call at m = B), then
    a draw from softmax(logits / T).  Each projection reads its own pre-drawn
    activation, as in a round."""

    def __init__(self, stack: Stack, temperature: float = 1.0):
        self.stack = stack
        cfg = self.cfg = stack.cfg
        dev = stack.device
        self.temperature = float(temperature)
        B, V, L = cfg.batch, cfg.vocab, stack.layers
        self.x, self.y = {}, {}
        for name, n, kin in cfg.layer_matrices():
            self.y[name] = torch.empty((B, n), dtype=torch.float16, device=dev)
            for l in range(L):
                mid = 1000 * (l + 1) + ["qkv", "o", "gate_up", "down"].index(name)
                self.x[(l, name)] = synth.normal_f16((B, kin), 1.0, synth.stream_seed(cfg.seed, _XDIRECT, mid), dev)
        if cfg.lm_head:
            self.x[(L, "lm_head")] = synth.normal_f16((B, cfg.hidden), 1.0, synth.stream_seed(cfg.seed, _XDIRECT), dev)
            self.logits = torch.empty((B, V), dtype=torch.float32, device=dev)
        else:
            self.logits = synth.normal_f32((B, V), 2.0, synth.stream_seed(cfg.seed, _BONUS), dev)
        self.u = torch.zeros((B, 1), dtype=torch.int32, device=dev)
        self.n_accepted = torch.zeros((B,), dtype=torch.int32, device=dev)
        self.token = torch.zeros((B,), dtype=torch.int32, device=dev)
        self.graph = None

    def run(self):
        st, cfg = self.stack, self.cfg
        for l in range(st.layers):
            for name, _, _ in cfg.layer_matrices():
                st.verify_gemm((l, name), self.x[(l, name)], self.y[name])
        if cfg.lm_head:
            st.verify_gemm((cfg.layers, "lm_head"), self.x[(st.layers, "lm_head")], self.logits)
        B, V = cfg.batch, cfg.vocab
        sq.sq_spec_accept(None, self.logits.view(B, 1, V), None, self.u, self.temperature,
                          n_accepted=self.n_accepted, next_token=self.token)

    def capture(self):
        self.run()
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            self.run()
        torch.cuda.synchronize()
        self.graph = g
        return g

    def replay(self):
        self.graph.replay()


def round_uniforms(cfg: Config, rounds: int, device):
    """Per-round uniforms: u_draft [R][k][B] and u_accept [R][B][k+1]."""
    B, k = cfg.batch, cfg.k
    ud = synth.uniform_u24((rounds, k, B), synth.stream_seed(cfg.seed, _UD), device)
    ua = synth.uniform_u24((rounds, B, k + 1), synth.stream_seed(cfg.seed, _UA), device)
    return ud, ua
