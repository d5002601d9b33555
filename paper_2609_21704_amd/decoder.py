"""SpecQuant rounds through a full decoder with a key/value cache.

The weight-streaming stack of ``rounds`` reads a fresh activation per
projection.  Here the same projections sit inside Qwen2.5-shaped decoder
layers (the model family of SS IV): the token embedding, per layer RMSNorm ->
q|k|v (+ bias) -> RoPE -> causal grouped-query attention over the cache -> o
-> residual -> RMSNorm -> gate|up -> SiLU . up -> down -> residual, then the
final RMSNorm and the LM head.  A round drafts k tokens with the quantized
copy (SS III-D.2), verifies the block with the FP16 parent (SS III-D.3),
accepts or corrects (SS III-D.4) and commits: the emitted tokens are
appended, and the sequence restarts at the emitted token, which rolls both
caches back to the accepted prefix by moving the position alone.

Every step runs in the library's HIP kernels; torch holds the buffers, and a
whole round can be captured as one HIP graph because all positions and
tokens live on the device.

Block layout per pass (b sequences, rows_per_seq rows each, rows at
pos_base + offset + j):
  draft step 0:   the previous token and the pending one at P-1, P (the entry
                  at P-1 is recomputed; it is missing after a round that
                  accepted every draft)
  draft step i:   draft i-1 at P+i
  verification:   the pending token and the k drafts at P .. P+k

Synthetic parameters (no checkpoints): the projection matrices are those of
``rounds.Stack`` (N(0, 0.02)); the embedding is N(0, 0.02), the norm weights
N(1, 0.02) and the q|k|v biases N(0, 0.02), all fp16, shared unquantized by
the draft copy.
"""
from __future__ import annotations

import dataclasses

import torch

from . import _lib as sq
from . import synth
from .configs import HEAD_DIM, Config
from .rounds import Stack, round_uniforms  # noqa: F401  (round_uniforms: per-round uniforms, same layout)

EPS = 1e-6
THETA = 1e6
# tensor ids for synth.stream_seed (distinct from those of rounds)
_EMBED, _NORM_IN, _NORM_POST, _NORM_FINAL, _BIAS, _PROMPT = range(20, 26)


class DecoderWeights:
    """The FP16 parent and its quantized draft copy (``Stack``) plus the
    embedding, norms and biases they share."""

    def __init__(self, cfg: Config, device, layers: int | None = None, variant: str | None = None,
                 stack: Stack | None = None):
        cfg = dataclasses.replace(cfg, lm_head=True)
        self.cfg = cfg
        self.device = dev = torch.device(device)
        if stack is not None:  # reuse the matrices of an existing stack (with its LM head and FP16 copies)
            if not stack.cfg.lm_head or not stack.w16:
                raise ValueError("the stack needs its LM head and its FP16 matrices")
            self.stack = stack
        else:
            self.stack = Stack(cfg, dev, variant=variant, layers=layers)
        self.layers = self.stack.layers
        H = cfg.hidden
        n_qkv = cfg.q_dim + 2 * cfg.kv_dim
        s = cfg.seed
        self.embed = synth.normal_f16((cfg.vocab, H), 0.02, synth.stream_seed(s, _EMBED), dev)
        self.final_norm = (synth.normal_f32((H,), 0.02, synth.stream_seed(s, _NORM_FINAL), dev) + 1.0).half()
        self.in_norm, self.post_norm, self.qkv_bias = [], [], []
        for l in range(self.layers):
            self.in_norm.append((synth.normal_f32((H,), 0.02, synth.stream_seed(s, _NORM_IN, l), dev) + 1.0).half())
            self.post_norm.append(
                (synth.normal_f32((H,), 0.02, synth.stream_seed(s, _NORM_POST, l), dev) + 1.0).half())
            self.qkv_bias.append(synth.normal_f16((n_qkv,), 0.02, synth.stream_seed(s, _BIAS, l), dev))

    def sibling(self, variant: str) -> "DecoderWeights":
        """The same parent, embedding, norms and biases with another draft copy."""
        other = DecoderWeights.__new__(DecoderWeights)
        other.__dict__.update(self.__dict__)
        other.stack = self.stack.sibling(variant)
        return other

    def params(self) -> dict:
        """Every parameter by the oracle's names (host float16 copies)."""
        p = {"embed": self.embed, "final_norm": self.final_norm,
             "lm_head": self.stack.w16[(self.cfg.layers, "lm_head")]}
        for l in range(self.layers):
            p[f"{l}.in_norm"] = self.in_norm[l]
            p[f"{l}.qkv_bias"] = self.qkv_bias[l]
            p[f"{l}.post_norm"] = self.post_norm[l]
            for name in ("qkv", "o", "gate_up", "down"):
                p[f"{l}.{name}"] = self.stack.w16[(l, name)]
        return {k: v.cpu().numpy() for k, v in p.items()}


class KVCache:
    """Keys [layers][rows][hkv][capacity][128] and position-minor values
    [layers][rows][hkv][128][capacity], fp16, one allocation each; k[l] and
    v[l] are the layer views the layer calls take."""

    def __init__(self, cfg: Config, layers: int, rows: int, capacity: int, device):
        if capacity % 64:
            raise ValueError("the cache capacity must be a multiple of 64")
        self.capacity = capacity
        self.k_all = torch.zeros((layers, rows, cfg.kv_heads, capacity, HEAD_DIM), dtype=torch.float16, device=device)
        self.v_all = torch.zeros((layers, rows, cfg.kv_heads, HEAD_DIM, capacity), dtype=torch.float16, device=device)
        self.k = [self.k_all[l] for l in range(layers)]
        self.v = [self.v_all[l] for l in range(layers)]


class _Buffers:
    """Activations of a pass of up to `rows` rows."""

    def __init__(self, cfg: Config, rows: int, device):
        H, I = cfg.hidden, cfg.intermediate
        n_qkv = cfg.q_dim + 2 * cfg.kv_dim
        f32, f16 = torch.float32, torch.float16
        self.h = torch.empty((rows, H), dtype=f32, device=device)
        self.x = torch.empty((rows, H), dtype=f16, device=device)
        self.qkv = torch.empty((rows, n_qkv), dtype=f32, device=device)
        self.q = torch.empty((rows, cfg.q_heads, HEAD_DIM), dtype=f16, device=device)
        self.a = torch.empty((rows, cfg.q_heads, HEAD_DIM), dtype=f16, device=device)
        self.y = torch.empty((rows, H), dtype=f32, device=device)
        self.gu = torch.empty((rows, 2 * I), dtype=f32, device=device)
        self.t = torch.empty((rows, I), dtype=f16, device=device)
        self.xf = torch.empty((rows, H), dtype=f16, device=device)


class SpecDecoder:
    """Speculative rounds of one batch of sequences through the decoder.

    With chains = c > 1 every sequence drafts c independent chains (its rows
    s c .. s c + c - 1 in every draft and verification pass, each with its own
    cache rows), and sq_spec_accept_multi accepts over them; the accepted
    chain's cache entries are then copied to the other chains and all of them
    restart from the emitted token."""

    def __init__(self, weights: DecoderWeights, batch: int | None = None, k: int | None = None,
                 capacity: int = 1024, temperature: float = 1.0, history: int = 4096, keep_pq: bool = False,
                 chains: int = 1, fuse: bool = True):
        self.w = weights
        cfg = self.cfg = weights.cfg
        dev = self.device = weights.device
        self.B = B = cfg.batch if batch is None else batch
        self.c = c = int(chains)
        self.R = R = B * c  # rows of a draft step: one per chain
        self.k = k = cfg.k if k is None else k
        self.T = float(temperature)
        V = cfg.vocab
        L = weights.layers
        if R * 2 > 64:
            raise ValueError("draft step 0 runs 2 rows per chain; a pass takes at most 64 rows")
        if R * (k + 1) > 64:
            raise ValueError("the verification pass takes at most 64 rows")
        self.dcache = KVCache(cfg, L, R, capacity, dev)
        self.pcache = KVCache(cfg, L, R, capacity, dev)
        self.capacity = capacity
        self.buf = _Buffers(cfg, 64, dev)  # the largest pass: 64 rows (verification, prefill chunks)
        i32, f32 = torch.int32, torch.float32
        self.pos_base = torch.zeros((R,), dtype=i32, device=dev)
        self.pending = torch.zeros((R,), dtype=i32, device=dev)
        self.prev = torch.zeros((R,), dtype=i32, device=dev)
        self.draft_tokens = torch.zeros((k, R), dtype=i32, device=dev)      # [k][B][c]
        self.draft_logits = torch.empty((k, R, V), dtype=f32, device=dev)   # [k][B][c][V]
        self.target_logits = torch.empty((R, k + 1, V), dtype=f32, device=dev)  # [B][c][k+1][V]
        self.u_draft = torch.zeros((k, R), dtype=i32, device=dev)
        self.u_accept = torch.zeros((B, c * k + 1), dtype=i32, device=dev)
        self.n_accepted = torch.zeros((B,), dtype=i32, device=dev)
        self.next_token = torch.zeros((B,), dtype=i32, device=dev)
        self.chain = torch.zeros((B,), dtype=i32, device=dev)
        self.scratch_n = torch.zeros((R,), dtype=i32, device=dev)
        self.out_tokens = torch.zeros((B, history), dtype=i32, device=dev)
        self.out_len = torch.zeros((B,), dtype=i32, device=dev)
        self.status = torch.zeros((1,), dtype=i32, device=dev)
        self.keep_pq = keep_pq
        self.attn_hook = None  # called as hook(True / False, rows_per_seq, offset) around each attention call
        if keep_pq:
            self.q_draft = torch.empty((k, R, V), dtype=f32, device=dev)   # draft-step distributions
            self.q_out = torch.empty((k, R, V), dtype=f32, device=dev)
            self.p_out = torch.empty((R, k + 1, V), dtype=f32, device=dev)
        self.graph = None
        self.fuse = fuse

    # ------------------------------------------------------------- passes
    def _linear(self, draft: bool, key, x, y):
        st = self.w.stack
        if draft:
            st.draft_gemv(key, x, y)
        else:
            st.verify_gemm(key, x, y)

    def _norm_linear(self, draft: bool, key, h, norm_w, delta, x, y, group: int = 1):
        """y = f16(rmsnorm(h [+ delta])) . W^T: in one launch where the projection
        normalises its own input rows (no pending delta), else the residual add
        + norm into x and the plain projection (the same bits either way)."""
        if delta is None and self.fuse:
            st = self.w.stack
            done = (st.draft_gemv_rmsnorm if draft else st.verify_gemm_rmsnorm)(key, h, norm_w, EPS, group, y)
            if done:
                return
        sq.sq_add_rmsnorm_f16(h, norm_w, EPS, delta=delta, group=group, x=x)
        self._linear(draft, key, x, y)

    def _residual_linear(self, draft: bool, key, x, h, y):
        """h += x . W^T where the projection adds into its output (returns None),
        else y = x . W^T, returned as the delta the next norm adds."""
        if self.fuse:
            st = self.w.stack
            if (st.draft_gemv_acc if draft else st.verify_gemm_acc)(key, x, h):
                return None
        self._linear(draft, key, x, y)
        return y

    def forward(self, draft: bool, first, rest, rps: int, offset: int, logits, last_only: bool,
                len_bound: int | None = None):
        """One pass of the block (first [R], rest [rps-1][R], R = batch x
        chains) at positions pos_base + offset + j through the draft (or
        parent) model, writing its cache entries; logits [R * (1 or rps)][V]
        f32 out."""
        cfg, w, b = self.cfg, self.w, self.buf
        M = self.R * rps
        if M > b.h.shape[0]:
            raise ValueError("a pass takes at most 64 rows")
        cache = self.dcache if draft else self.pcache
        lb = self.capacity if len_bound is None else len_bound
        h, x, qkv, q, a, y, gu, t = (b.h[:M], b.x[:M], b.qkv[:M], b.q[:M], b.a[:M], b.y[:M], b.gu[:M], b.t[:M])
        sq.sq_embed_block_f16(w.embed, first, rest, h=h, status=self.status)
        delta = None  # a projection output not yet added into h
        for l in range(w.layers):
            self._norm_linear(draft, (l, "qkv"), h, w.in_norm[l], delta, x, qkv)
            if not (self.fuse and self.attn_hook is None and
                    sq.sq_rope_attention_f16(qkv, w.qkv_bias[l], self.pos_base, offset, rps, cfg.q_heads,
                                             cache.k[l], cache.v[l], a, len_bound=lb, theta=THETA,
                                             status=self.status)):
                sq.sq_rope_kv_f16(qkv, w.qkv_bias[l], self.pos_base, offset, rps, cfg.q_heads, cache.k[l],
                                  cache.v[l], len_bound=lb, theta=THETA, q_out=q, status=self.status)
                if self.attn_hook:
                    self.attn_hook(True, rps, offset)
                sq.sq_attention_f16(q, cache.k[l], cache.v[l], self.pos_base, offset, rps, len_bound=lb, out=a)
                if self.attn_hook:
                    self.attn_hook(False, rps, offset)
            delta = self._residual_linear(draft, (l, "o"), a.view(M, cfg.q_dim), h, y)
            if not (draft and delta is None and self.fuse and
                    w.stack.draft_gemv_rmsnorm_silu((l, "gate_up"), h, w.post_norm[l], EPS, t)):
                self._norm_linear(draft, (l, "gate_up"), h, w.post_norm[l], delta, x, gu)
                sq.sq_silu_mul_f16(gu, t)
            delta = self._residual_linear(draft, (l, "down"), t, h, y)
        group = rps if last_only else 1
        xf = b.xf[:M // group]
        self._norm_linear(draft, (cfg.layers, "lm_head"), h, w.final_norm, delta, xf, logits, group=group)

    def prefill(self, prompt: torch.Tensor, chunk: int | None = None, models=(True, False), lengths=None):
        """Feed prompt [B][Lp] (int32) but its last token to both models
        (every chain of a sequence gets the sequence's prompt); the last token
        becomes the pending one at position Lp - 1.  `models` lists the passes
        to run (True: the draft, False: the parent).

        With lengths [B] (2 <= lengths[s] <= Lp) the prompts are ragged:
        sequence s is prompt[s][:lengths[s]], and the tokens past it are
        padding.  Every row is fed Lp - 1 tokens; a short row's entries from
        its last prompt position on are rewritten before any row attends to
        them, as a rolled-back draft block's are, so the padding is never
        read."""
        B, Lp = prompt.shape
        if B != self.B or Lp < 2 or Lp > self.capacity:
            raise ValueError("prompt must be [batch][2 .. capacity]")
        if lengths is None:
            lens = torch.full((B,), Lp, dtype=torch.int64)
        else:
            lens = torch.as_tensor(lengths, dtype=torch.int64).cpu()
            if lens.shape != (B,) or int(lens.min()) < 2 or int(lens.max()) > Lp:
                raise ValueError("lengths must be [batch] in 2 .. prompt length")
        host = prompt.to(device="cpu", dtype=torch.int32).repeat_interleave(self.c, dim=0)
        lens = lens.repeat_interleave(self.c)
        rows = torch.arange(self.R)
        last, before = host[rows, lens - 1].contiguous(), host[rows, lens - 2].contiguous()
        prompt = host.to(self.device)
        R = self.R
        self.pos_base.zero_()
        V = self.cfg.vocab
        for draft in models:
            c = max(1, min(chunk or 64, 64 // R))
            for s in range(0, Lp - 1, c):
                n = min(c, Lp - 1 - s)
                first = prompt[:, s].contiguous()
                rest = prompt[:, s + 1:s + n].t().contiguous() if n > 1 else None
                logits = torch.empty((R * n, V), dtype=torch.float32, device=self.device)
                self.forward(draft, first, rest, n, s, logits, last_only=False, len_bound=s + n)
        self.pos_base.copy_((lens - 1).to(torch.int32))
        self.pending.copy_(last)
        self.prev.copy_(before)
        self.out_len.zero_()

    # -------------------------------------------------------------- round
    def draft_step(self, i: int):
        R, V = self.R, self.cfg.vocab
        if i == 0:
            self.forward(True, self.prev, self.pending.view(1, R), 2, -1, self.draft_logits[0], last_only=True)
        else:
            self.forward(True, self.draft_tokens[i - 1], None, 1, i, self.draft_logits[i], last_only=True)
        p_out = self.q_draft[i].view(R, 1, V) if self.keep_pq and self.T > 0 else None
        sq.sq_spec_accept(None, self.draft_logits[i].view(R, 1, V), None, self.u_draft[i].view(R, 1), self.T,
                          n_accepted=self.scratch_n, next_token=self.draft_tokens[i], p_out=p_out)

    def verify(self):
        R, k, V = self.R, self.k, self.cfg.vocab
        self.forward(False, self.pending, self.draft_tokens, k + 1, 0, self.target_logits.view(R * (k + 1), V),
                     last_only=False)

    def accept_and_commit(self):
        keep = self.keep_pq and self.T > 0
        B, c, k, V = self.B, self.c, self.k, self.cfg.vocab
        if c == 1:
            sq.sq_spec_accept(self.draft_logits, self.target_logits, self.draft_tokens, self.u_accept, self.T,
                              n_accepted=self.n_accepted, next_token=self.next_token,
                              q_out=self.q_out if keep else None, p_out=self.p_out if keep else None)
            sq.sq_spec_commit(self.n_accepted, self.next_token, self.draft_tokens, self.pending, self.prev,
                              self.pos_base, out_tokens=self.out_tokens, out_len=self.out_len, status=self.status)
            return
        sq.sq_spec_accept_multi(self.draft_logits.view(k, B, c, V), self.target_logits.view(B, c, k + 1, V),
                                self.draft_tokens.view(k, B, c), self.u_accept, self.T, n_accepted=self.n_accepted,
                                next_token=self.next_token, chain=self.chain,
                                q_out=self.q_out.view(k, B, c, V) if keep else None,
                                p_out=self.p_out.view(B, c, k + 1, V) if keep else None)
        # the accepted chain's entries to the other chains: the parent's at P .. P + n,
        # the draft's at P - 1 .. P + n - 1
        sq.sq_kv_adopt_f16(self.pcache.k_all, self.pcache.v_all, B, c, self.chain, self.n_accepted, self.pos_base,
                           0, 0)
        sq.sq_kv_adopt_f16(self.dcache.k_all, self.dcache.v_all, B, c, self.chain, self.n_accepted, self.pos_base,
                           -1, -1)
        sq.sq_spec_commit_multi(self.n_accepted, self.next_token, self.chain, self.draft_tokens, c, self.pending,
                                self.prev, self.pos_base, out_tokens=self.out_tokens, out_len=self.out_len,
                                status=self.status)

    def run(self):
        for i in range(self.k):
            self.draft_step(i)
        self.verify()
        self.accept_and_commit()

    def set_uniforms(self, u_draft: torch.Tensor, u_accept: torch.Tensor):
        self.u_draft.copy_(u_draft)
        self.u_accept.copy_(u_accept)

    def capture(self):
        """Capture one round as a HIP graph.  Runs one round eagerly first (it
        advances the sequences by one round), so that the library workspace
        has its final size before capture."""
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


class DirectDecoder(SpecDecoder):
    """Direct parent inference (SS III-D.5) through the decoder: one token per
    sequence and step from the FP16 parent alone (its pass at one row per
    sequence, a draw from softmax(logits / T) or the argmax, the commit).  The
    route of high-complexity prompts, and the plain-decoding baseline."""

    def __init__(self, weights: DecoderWeights, batch: int | None = None, capacity: int = 1024,
                 temperature: float = 1.0, history: int = 4096, fuse: bool = True):
        self.w = weights
        self.fuse = fuse
        cfg = self.cfg = weights.cfg
        dev = self.device = weights.device
        self.B = self.R = B = cfg.batch if batch is None else batch
        self.c, self.k = 1, 0
        self.T = float(temperature)
        if B > 64:
            raise ValueError("a parent pass takes at most 64 rows")
        self.dcache = None
        self.pcache = KVCache(cfg, weights.layers, B, capacity, dev)
        self.capacity = capacity
        self.buf = _Buffers(cfg, 64, dev)
        i32 = torch.int32
        self.pos_base = torch.zeros((B,), dtype=i32, device=dev)
        self.pending = torch.zeros((B,), dtype=i32, device=dev)
        self.prev = torch.zeros((B,), dtype=i32, device=dev)
        self.logits = torch.empty((B, cfg.vocab), dtype=torch.float32, device=dev)
        self.u = torch.zeros((B, 1), dtype=i32, device=dev)
        self.n_accepted = torch.zeros((B,), dtype=i32, device=dev)
        self.next_token = torch.zeros((B,), dtype=i32, device=dev)
        self.out_tokens = torch.zeros((B, history), dtype=i32, device=dev)
        self.out_len = torch.zeros((B,), dtype=i32, device=dev)
        self.status = torch.zeros((1,), dtype=i32, device=dev)
        self.keep_pq = False
        self.attn_hook = None
        self.graph = None

    def prefill(self, prompt: torch.Tensor, chunk: int | None = None, models=(False,), lengths=None):
        super().prefill(prompt, chunk, models=models, lengths=lengths)

    def set_uniforms(self, u: torch.Tensor, _unused=None):
        self.u.copy_(u.view(self.B, 1))

    def run(self):
        B, V = self.B, self.cfg.vocab
        self.forward(False, self.pending, None, 1, 0, self.logits, last_only=False)
        sq.sq_spec_accept(None, self.logits.view(B, 1, V), None, self.u, self.T, n_accepted=self.n_accepted,
                          next_token=self.next_token)
        sq.sq_spec_commit(self.n_accepted, self.next_token, None, self.pending, self.prev, self.pos_base,
                          out_tokens=self.out_tokens, out_len=self.out_len, status=self.status)


def synthetic_prompt(cfg: Config, batch: int, length: int, device) -> torch.Tensor:
    """Uniform random token ids [batch][length] from the config seed."""
    return synth.tokens((batch, length), cfg.vocab, synth.stream_seed(cfg.seed, _PROMPT, length), device)
