"""Oracle of the decoder step and of the speculative round with its cache --
test infrastructure only (same rules as the rest of ``oracle``).

SpecQuant (arXiv 2609.21704) drafts with a quantized parent (SS III-D.2),
verifies the drafted block with the FP16 parent (SS III-D.3), accepts or
corrects (SS III-D.4) and, after a rejection, removes the rest of the
speculative block and restarts from the first rejected token.  The paper
evaluates Qwen2.5 models (SS IV) and does not describe the layer; this module
composes the textbook operations of that family (``sq_decoder.c``) into one
decoder layer, the full forward pass, and the round with a key/value cache:

  h = embed[token]
  per layer:  x = f16(rmsnorm(h, w_in))
              q | k | v = x . Wqkv'^T + b_qkv,  q, k <- rope(q, k at position)
              cache[position] = (f16(k), f16(v));  a = f16(attention(f16(q), cache))
              h = h + a . Wo'^T
              x = f16(rmsnorm(h, w_post))
              h = h + f16(silu(x . Wg'^T) * (x . Wu'^T)) . Wd'^T
  logits = f16(rmsnorm(h, w_final)) . Wlm'^T

W' is the variant's matrix: the FP16 parent itself, or its INT4 / FP8 copy
made by this oracle's own quantizers.  Arithmetic is fp64; f16(.) marks where
a value becomes the binary16 input of the next operation (the projections take
binary16 activations, and the cache holds binary16 keys and values), rounded to
nearest-even.  The embedding, norms and biases are shared, unquantized, by all
variants.

The round (k drafts per sequence, position P of the pending token):
  draft step 0 feeds the previous token and the pending one (positions P-1, P;
  the entry at P-1 is recomputed, which fills it when the previous round
  accepted every draft), step i > 0 feeds draft i-1 at P+i; each step draws
  its draft from the last row's logits.  The parent feeds the pending token and
  the k drafts at P .. P+k.  After accepting n drafts and emitting the next
  token, the pending token is that next token at P+n+1: cache entries from that
  position on belong to the removed block and are never read again before being
  overwritten.

With c draft chains per sequence (spec_round_multi) the caches hold c rows per
sequence (row s c + j for chain j, each started from the sequence's prompt);
every chain drafts its own tokens, the parent verifies all of them, acceptance
walks the chains' prefix tree (``multi_accept``), and the accepted chain's new
entries are copied to the other chains before all of them restart.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

from . import (attention, dequant_fp8, dequant_int4, multi_accept, quantize_fp8_e4m3, quantize_int4_g128, rmsnorm,
               rope, silu_mul, spec_accept)

HEAD_DIM = 128
MATRICES = ("qkv", "o", "gate_up", "down")


def f16(a) -> np.ndarray:
    """Round to binary16, nearest-even (numpy's direct double -> half conversion)."""
    return np.asarray(a, np.float64).astype(np.float16)


@dataclass
class Dims:
    layers: int
    hidden: int
    inter: int
    q_heads: int
    kv_heads: int
    vocab: int
    eps: float = 1e-6
    theta: float = 1e6

    @property
    def q_dim(self) -> int:
        return self.q_heads * HEAD_DIM

    @property
    def kv_dim(self) -> int:
        return self.kv_heads * HEAD_DIM


class Model:
    """One variant of the model: params maps names to float16 arrays
    ('embed' [V][H], 'final_norm' [H], 'lm_head' [V][H], and per layer l
    'l.in_norm', 'l.qkv', 'l.qkv_bias', 'l.o', 'l.post_norm', 'l.gate_up',
    'l.down'); variant is 'f16', 'int4' or 'fp8'."""

    def __init__(self, dims: Dims, params: dict, variant: str):
        if variant not in ("f16", "int4", "fp8"):
            raise ValueError(variant)
        self.dims = dims
        self.params = params
        self.variant = variant
        self._w = {}

    def vec(self, name: str) -> np.ndarray:
        return np.asarray(self.params[name], np.float16).astype(np.float64)

    def weight(self, name: str) -> np.ndarray:
        """fp64 W' of a matrix for this variant (kept after the first use)."""
        w = self._w.get(name)
        if w is None:
            w16 = np.asarray(self.params[name], np.float16)
            if self.variant == "f16":
                w = w16.astype(np.float64)
            elif self.variant == "int4":
                codes, scales, zeros = quantize_int4_g128(w16)
                w = dequant_int4(codes, scales, zeros, w16.shape[1])
            else:
                codes, scales = quantize_fp8_e4m3(w16)
                w = dequant_fp8(codes, scales)
            self._w[name] = w
        return w

    def linear(self, name: str, x16) -> np.ndarray:
        x = np.asarray(x16, np.float16)
        return x.astype(np.float64) @ self.weight(name).T


class Cache:
    """Keys and values of one model: [layer][sequence][kv head][position][128],
    binary16 values held in fp64; unwritten entries are NaN."""

    def __init__(self, dims: Dims, batch: int, capacity: int):
        shape = (dims.layers, batch, dims.kv_heads, capacity, HEAD_DIM)
        self.k = np.full(shape, np.nan)
        self.v = np.full(shape, np.nan)
        self.capacity = capacity


def forward(model: Model, cache: Cache, tokens, positions, record: dict | None = None) -> np.ndarray:
    """Run the rows tokens [B][r] at positions [B][r] through the model, writing
    their keys and values into the cache; returns the logits [B][r][V] (fp64).
    Row j of sequence b attends to that sequence's positions 0 .. positions[b][j].
    If record is a dict, the intermediate tensors of every layer are stored in it."""
    d = model.dims
    tokens = np.asarray(tokens, np.int64)
    positions = np.asarray(positions, np.int64)
    B, r = tokens.shape
    if positions.shape != (B, r):
        raise ValueError("positions must match tokens")
    if positions.min() < 0 or positions.max() >= cache.capacity:
        raise ValueError("position outside the cache")
    D, hq, hkv = HEAD_DIM, d.q_heads, d.kv_heads
    h = np.asarray(model.params["embed"], np.float16)[tokens.reshape(-1)].astype(np.float64)
    flat_pos = positions.reshape(-1)
    for l in range(d.layers):
        x = f16(rmsnorm(h, model.vec(f"{l}.in_norm"), d.eps))
        qkv = model.linear(f"{l}.qkv", x) + model.vec(f"{l}.qkv_bias")
        q = rope(qkv[:, :d.q_dim].reshape(B * r, hq, D), flat_pos, d.theta)
        k = rope(qkv[:, d.q_dim:d.q_dim + d.kv_dim].reshape(B * r, hkv, D), flat_pos, d.theta)
        v = qkv[:, d.q_dim + d.kv_dim:].reshape(B * r, hkv, D)
        q16, k16, v16 = f16(q), f16(k), f16(v)
        for b in range(B):
            for j in range(r):
                cache.k[l, b, :, positions[b, j], :] = k16[b * r + j].astype(np.float64)
                cache.v[l, b, :, positions[b, j], :] = v16[b * r + j].astype(np.float64)
        a = np.zeros((B * r, hq, D))
        for b in range(B):
            length = int(positions[b].max()) + 1
            a[b * r:(b + 1) * r] = attention(q16[b * r:(b + 1) * r].astype(np.float64),
                                             cache.k[l, b, :, :length], cache.v[l, b, :, :length], positions[b])
        a16 = f16(a).reshape(B * r, d.q_dim)
        o = model.linear(f"{l}.o", a16)
        h = h + o
        x2 = f16(rmsnorm(h, model.vec(f"{l}.post_norm"), d.eps))
        gu = model.linear(f"{l}.gate_up", x2)
        t16 = f16(silu_mul(gu))
        dn = model.linear(f"{l}.down", t16)
        if record is not None:
            record[l] = {"x": x, "qkv": qkv, "q16": q16, "k16": k16, "v16": v16, "a16": a16, "o": o,
                         "x2": x2, "gu": gu, "t16": t16, "down": dn, "h_mid": h.copy()}
        h = h + dn
        if record is not None:
            record[l]["h_out"] = h.copy()
    xf = f16(rmsnorm(h, model.vec("final_norm"), d.eps))
    logits = model.linear("lm_head", xf)
    if record is not None:
        record["final_x"] = xf
    return logits.reshape(B, r, d.vocab)


@dataclass
class SpecState:
    """Per sequence: position of the pending token, the pending token, the token
    before it, and every token emitted so far."""
    pos: np.ndarray
    pending: np.ndarray
    prev: np.ndarray
    emitted: list = field(default_factory=list)


def prefill(models, caches, prompt) -> SpecState:
    """Feed prompt [B][Lp] (Lp >= 2) but its last token to every model; the last
    prompt token becomes the pending token at position Lp - 1."""
    prompt = np.asarray(prompt, np.int64)
    B, Lp = prompt.shape
    if Lp < 2:
        raise ValueError("the prompt needs at least two tokens")
    pos = np.broadcast_to(np.arange(Lp - 1), (B, Lp - 1))
    for m, c in zip(models, caches):
        forward(m, c, prompt[:, :Lp - 1], pos)
    return SpecState(pos=np.full(B, Lp - 1, np.int64), pending=prompt[:, Lp - 1].copy(),
                     prev=prompt[:, Lp - 2].copy(), emitted=[[] for _ in range(B)])


def commit(state: SpecState, n_accepted, next_token, drafts) -> None:
    """Append the accepted drafts and the next token; the next token becomes the
    pending one at P + n + 1 (the rest of the block is removed).  A sequence
    whose round had no distribution (n = -1) keeps its state."""
    drafts = np.asarray(drafts, np.int64)  # [k][B]
    for b in range(len(state.pos)):
        n = int(n_accepted[b])
        if n < 0:
            continue
        state.emitted[b].extend(int(t) for t in drafts[:n, b])
        state.emitted[b].append(int(next_token[b]))
        state.prev[b] = drafts[n - 1, b] if n >= 1 else state.pending[b]
        state.pending[b] = int(next_token[b])
        state.pos[b] += n + 1


def spec_round(draft: Model, parent: Model, dcache: Cache, pcache: Cache, state: SpecState, k: int,
               u_draft, u_accept, temperature: float = 1.0) -> dict:
    """One round: k draft steps, the parent's pass over the block, accept /
    correct, commit.  u_draft [k][B], u_accept [B][k+1] (24-bit uniforms;
    None at temperature 0, where the rule is greedy)."""
    B = len(state.pos)
    P = state.pos.copy()
    if u_draft is not None:
        u_draft = np.asarray(u_draft, np.uint32).reshape(k, B)
    drafts, qlog = [], []
    for i in range(k):
        if i == 0:
            toks = np.stack([state.prev, state.pending], 1)
            pos = np.stack([P - 1, P], 1)
        else:
            toks = drafts[-1][:, None]
            pos = (P + i)[:, None]
        lg = forward(draft, dcache, toks, pos)[:, -1]
        lg32 = lg.astype(np.float32)
        qlog.append(lg32)
        u = None if u_draft is None else u_draft[i][:, None]
        _, tok, _, _ = spec_accept(None, lg32[:, None, :], None, u, temperature)
        drafts.append(tok.astype(np.int64))
    vt = np.concatenate([state.pending[:, None], np.stack(drafts, 1)], 1)
    vp = P[:, None] + np.arange(k + 1)[None, :]
    target = forward(parent, pcache, vt, vp).astype(np.float32)
    dl = np.stack(qlog, 0)
    dt = np.stack(drafts, 0)
    n_acc, nxt, _, _ = spec_accept(dl, target, dt.astype(np.int32), u_accept, temperature)
    commit(state, n_acc, nxt, dt)
    return {"draft_tokens": dt, "draft_logits": dl, "target_logits": target, "n_accepted": n_acc,
            "next_token": nxt, "positions": P}


def prefill_chains(models, caches, prompt, c: int) -> SpecState:
    """prefill with every sequence repeated for its c chains (cache rows s c + j)."""
    prompt = np.asarray(prompt, np.int64)
    st = prefill(models, caches, np.repeat(prompt, c, axis=0))
    B = prompt.shape[0]
    return SpecState(pos=st.pos[::c].copy(), pending=st.pending[::c].copy(), prev=st.prev[::c].copy(),
                     emitted=[[] for _ in range(B)])


def spec_round_multi(draft: Model, parent: Model, dcache: Cache, pcache: Cache, state: SpecState, c: int, k: int,
                     u_draft, u_accept, temperature: float = 1.0) -> dict:
    """One round with c chains per sequence: u_draft [k][B c] (each chain's own
    draws), u_accept [B][c k + 1]."""
    B = len(state.pos)
    R = B * c
    P = np.repeat(state.pos, c)
    prev, pend = np.repeat(state.prev, c), np.repeat(state.pending, c)
    if u_draft is not None:
        u_draft = np.asarray(u_draft, np.uint32).reshape(k, R)
    drafts, qlog = [], []
    for i in range(k):
        if i == 0:
            toks, pos = np.stack([prev, pend], 1), np.stack([P - 1, P], 1)
        else:
            toks, pos = drafts[-1][:, None], (P + i)[:, None]
        lg32 = forward(draft, dcache, toks, pos)[:, -1].astype(np.float32)
        qlog.append(lg32)
        u = None if u_draft is None else u_draft[i][:, None]
        _, tok, _, _ = spec_accept(None, lg32[:, None, :], None, u, temperature)
        drafts.append(tok.astype(np.int64))
    vt = np.concatenate([pend[:, None], np.stack(drafts, 1)], 1)
    target = forward(parent, pcache, vt, P[:, None] + np.arange(k + 1)[None, :]).astype(np.float32)
    V = target.shape[-1]
    dl = np.stack(qlog, 0).reshape(k, B, c, V)
    dt = np.stack(drafts, 0).reshape(k, B, c)
    n, nxt, ch = multi_accept(dl, target.reshape(B, c, k + 1, V), dt.astype(np.int32), u_accept, temperature)
    adopt(pcache, dcache, state.pos, n, ch, c)
    sel = np.zeros((k, B), np.int64)
    for s in range(B):
        if n[s] >= 0:
            sel[:, s] = dt[:, s, ch[s]]
    commit(state, n, nxt, sel)
    return {"draft_tokens": dt, "draft_logits": dl, "target_logits": target.reshape(B, c, k + 1, V),
            "n_accepted": n, "next_token": nxt, "chain": ch, "positions": P}


def adopt(pcache: Cache, dcache: Cache, pos, n, ch, c: int) -> None:
    """Copy the accepted chain's new entries to the other chains of each
    sequence: the parent's at P .. P + n, the draft's at P - 1 .. P + n - 1."""
    for s in range(len(pos)):
        if n[s] < 0:
            continue
        src = s * c + int(ch[s])
        P = int(pos[s])
        for j in range(c):
            dst = s * c + j
            if dst == src:
                continue
            for cache, lo, hi in ((pcache, P, P + n[s]), (dcache, max(P - 1, 0), P + n[s] - 1)):
                cache.k[:, dst, :, lo:hi + 1] = cache.k[:, src, :, lo:hi + 1]
                cache.v[:, dst, :, lo:hi + 1] = cache.v[:, src, :, lo:hi + 1]
