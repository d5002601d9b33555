"""The SpecQuant execution pipeline (SS III-D): complexity assessment, then
speculative rounds with the routed draft or direct parent decoding.

One FP16 parent is resident with the quantized copies derived from it (SS
III-A): INT4 g128 (Q4) and FP8 e4m3 (Q8) share the parent's matrices,
embedding, norms and biases.  `Router` assigns each request a route
("int4", "fp8" or "f16"); requests of one route are batched, their ragged
prompts prefilled together, and their rounds run as captured HIP graphs
until every sequence has its tokens:

  int4, fp8   SpecDecoder with that draft: k drafts, one parent pass over the
              block, accept or correct, commit (SS III-D.2 to III-D.4)
  f16         DirectDecoder: the parent alone, one token per round (SS III-D.5)

Placement (SS III-C).  The parent always stays on the GPU.  A draft copy is
made resident only when it fits in the HBM left after the parent, the caches
and a margin; a route whose draft is absent is served by the other draft if
that one is resident, else by the parent directly.  The paper instead runs a
draft that does not fit on the host CPU; with 288 GB of HBM both drafts fit
beside the parent of every Qwen2.5 shape up to 72B, so no host path exists.
"""
from __future__ import annotations

import dataclasses
import time

import torch

from . import synth
from .configs import HEAD_DIM, Config
from .decoder import DecoderWeights, DirectDecoder, SpecDecoder
from .router import ROUTES, Router, features, hash_tokenize

_U_DRAFT, _U_ACCEPT, _U_DIRECT = 140, 141, 142  # ids for synth.stream_seed


def weight_bytes(cfg: Config, layers: int | None = None) -> dict:
    """HBM bytes of the parent (FP16 matrices, embedding, norms, biases) and
    of each draft copy's matrices."""
    L = cfg.layers if layers is None else layers
    cfg = dataclasses.replace(cfg, lm_head=True)
    mats = [(n, k) for (l, name, n, k) in cfg.matrices() if l < L or name == "lm_head"]
    nk = sum(n * k for n, k in mats)
    extra = cfg.vocab * cfg.hidden * 2 + (2 * L + 1) * cfg.hidden * 2 + L * (cfg.q_dim + 2 * cfg.kv_dim) * 2
    return {
        "f16": 2 * nk + extra,
        "int4": nk // 2 + sum(n * (k // 128) * 4 for n, k in mats),
        "fp8": nk + sum(4 * n for n, _ in mats),
    }


def cache_bytes(cfg: Config, layers: int, rows: int, capacity: int) -> int:
    """Keys and values of one model's cache: fp16, per layer, row, kv head and position."""
    return 2 * layers * rows * cfg.kv_heads * capacity * HEAD_DIM * 2


def placement(cfg: Config, free_bytes: int, batch: int, capacity: int, k: int, layers: int | None = None,
              margin: float = 0.1) -> dict:
    """Which variants are resident, given the device's free HBM: the parent
    and its direct-decoding cache first (required), then the INT4 draft with
    the caches of its decoder, then the FP8 draft with its own.  `margin` of
    free_bytes stays unplanned (activations, workspace, allocator slack).
    Returns {"resident": [...], "route_to": {route: served_by}, "bytes": {...}}."""
    L = cfg.layers if layers is None else layers
    w = weight_bytes(cfg, L)
    budget = int(free_bytes * (1.0 - margin))
    direct = w["f16"] + cache_bytes(cfg, L, batch, capacity)
    if direct > budget:
        raise MemoryError(f"the FP16 parent and its cache need {direct} bytes; {budget} are available")
    used, resident = direct, ["f16"]
    spec_cache = 2 * cache_bytes(cfg, L, batch, capacity)  # draft and parent caches of one SpecDecoder
    for v in ("int4", "fp8"):
        if used + w[v] + spec_cache <= budget:
            used += w[v] + spec_cache
            resident.append(v)
    route_to = {}
    for r in ROUTES:
        if r in resident:
            route_to[r] = r
        else:
            other = "fp8" if r == "int4" else "int4"
            route_to[r] = other if other in resident else "f16"
    return {"resident": resident, "route_to": route_to, "bytes": {"planned": used, "budget": budget, **w}}


@dataclasses.dataclass
class Result:
    route: str           # the route the router chose
    served_by: str       # the variant that decoded it (differs when that draft is not resident)
    prompt_tokens: int
    tokens: list         # the generated token ids


class Engine:
    """Routes requests to the speculative INT4 / FP8 decoders or to direct
    FP16 decoding, and generates their tokens on one GPU."""

    def __init__(self, cfg: Config, device, layers: int | None = None, k: int | None = None, batch: int = 4,
                 capacity: int = 1024, temperature: float = 0.0, router: Router | None = None,
                 chains: int = 1, free_bytes: int | None = None, seed: int | None = None,
                 parent: DecoderWeights | None = None, timed: bool = False):
        """`parent`: existing FP16 parent weights (with one draft copy) to serve
        from instead of building new ones.  `timed`: synchronise around each
        batch's prefill and rounds and add their wall time to `seconds`."""
        self.cfg = cfg
        self.device = torch.device(device)
        self.k = cfg.k if k is None else k
        self.batch, self.capacity, self.T, self.chains = batch, capacity, float(temperature), chains
        self.router = router or Router()
        self.seed = cfg.seed if seed is None else seed
        L = cfg.layers if layers is None else layers
        if free_bytes is None:
            free_bytes = torch.cuda.mem_get_info(self.device)[0]
        self.plan = placement(cfg, free_bytes, batch * chains, capacity, self.k, L)
        resident = self.plan["resident"]
        if parent is None:
            first = "int4" if "int4" in resident else ("fp8" if "fp8" in resident else "none")
            parent = DecoderWeights(cfg, self.device, layers=L, variant=first)
        elif parent.layers != L or parent.cfg.vocab != cfg.vocab or parent.cfg.hidden != cfg.hidden:
            raise ValueError("the parent weights do not have this configuration's shape")
        first = parent.stack.variant
        self.weights = {"f16": parent}
        for v in ("int4", "fp8"):
            if v in resident:
                self.weights[v] = parent if v == first else parent.sibling(v)
        self.decoders = {}
        self.rounds = {r: 0 for r in ROUTES}   # rounds run per variant
        self.emitted = {r: 0 for r in ROUTES}  # tokens kept per variant
        self._batches = 0
        self.timed = timed
        self.seconds = {(r, phase): 0.0 for r in ROUTES for phase in ("prefill", "rounds")}

    def decoder(self, variant: str):
        if variant not in self.decoders:
            w = self.weights[variant]
            if variant == "f16":
                self.decoders[variant] = DirectDecoder(w, batch=self.batch, capacity=self.capacity,
                                                       temperature=self.T, history=self.capacity)
            else:
                self.decoders[variant] = SpecDecoder(w, batch=self.batch, k=self.k, capacity=self.capacity,
                                                     temperature=self.T, chains=self.chains,
                                                     history=self.capacity)
        return self.decoders[variant]

    def tokenize(self, prompt) -> list:
        return hash_tokenize(prompt, self.cfg.vocab) if isinstance(prompt, str) else [int(t) for t in prompt]

    def classify(self, prompt) -> str:
        """The route of one request: text is scored on its own features; a
        token list only has its length, so its syntax and entity terms are 0."""
        if isinstance(prompt, str):
            return self.router.classify(features(prompt, len(self.tokenize(prompt)), self.cfg.vocab))
        return self.router.classify(features("", len(prompt)))

    def generate(self, prompts, max_new: int, routes=None) -> list[Result]:
        """Generate max_new tokens for each prompt (a text or a list of token
        ids, at least two tokens); `routes` overrides the router per request."""
        if max_new < 1:
            raise ValueError("max_new must be at least 1")
        toks = [self.tokenize(p) for p in prompts]
        chosen = list(routes) if routes is not None else [self.classify(p) for p in prompts]
        if len(chosen) != len(toks) or any(r not in ROUTES for r in chosen):
            raise ValueError(f"one route per prompt, each one of {ROUTES}")
        for t in toks:
            if len(t) < 2 or len(t) + max_new + self.k + 1 > self.capacity:
                raise ValueError(f"a prompt of {len(t)} tokens does not fit {max_new} new tokens in "
                                 f"{self.capacity} cache positions")
            if min(t) < 0 or max(t) >= self.cfg.vocab:
                raise ValueError("token ids must lie in [0, vocab)")
        out = [None] * len(toks)
        for variant in ROUTES:
            idx = [i for i, r in enumerate(chosen) if self.plan["route_to"][r] == variant]
            for s in range(0, len(idx), self.batch):
                part = idx[s:s + self.batch]
                gen = self._run_batch(variant, [toks[i] for i in part], max_new)
                for i, g in zip(part, gen):
                    out[i] = Result(route=chosen[i], served_by=variant, prompt_tokens=len(toks[i]), tokens=g)
        return out

    def _uniforms(self, variant: str, r: int):
        B, k, c = self.batch, self.k, self.chains
        ids = (self._batches, r)
        if variant == "f16":
            return synth.uniform_u24((B, 1), synth.stream_seed(self.seed, _U_DIRECT, *ids), self.device), None
        return (synth.uniform_u24((k, B * c), synth.stream_seed(self.seed, _U_DRAFT, *ids), self.device),
                synth.uniform_u24((B, c * k + 1), synth.stream_seed(self.seed, _U_ACCEPT, *ids), self.device))

    def _run_batch(self, variant: str, toks: list, max_new: int) -> list:
        dec = self.decoder(variant)
        n = len(toks)
        rows = toks + [toks[0]] * (self.batch - n)  # idle rows repeat the first prompt
        Lp = max(len(t) for t in rows)
        prompt = torch.zeros((self.batch, Lp), dtype=torch.int32)
        for i, t in enumerate(rows):
            prompt[i, :len(t)] = torch.tensor(t, dtype=torch.int32)
        t0 = self._clock()
        dec.prefill(prompt, lengths=[len(t) for t in rows])
        t1 = self._clock()
        per_round = 1 if variant == "f16" else self.k + 1
        r = 0
        while True:
            dec.set_uniforms(*self._uniforms(variant, r))
            if dec.graph is None:
                dec.capture()  # runs this round eagerly, then records the graph
            else:
                dec.replay()
            r += 1
            # every round emits at least one token per sequence: check only once enough rounds may have run
            if r * per_round >= max_new and int(dec.out_len[:n].min().item()) >= max_new:
                break
            if r > max_new:
                raise RuntimeError("a round emitted no token")
        t2 = self._clock()
        if self.timed:
            self.seconds[(variant, "prefill")] += t1 - t0
            self.seconds[(variant, "rounds")] += t2 - t1
        if int(dec.status.item()) != 0:
            raise RuntimeError(f"device status flags {int(dec.status.item())} raised")
        self._batches += 1
        self.rounds[variant] += r
        self.emitted[variant] += n * max_new
        return dec.out_tokens[:n, :max_new].cpu().tolist()

    def _clock(self) -> float:
        if not self.timed:
            return 0.0
        torch.cuda.synchronize(self.device)
        return time.perf_counter()

    def stats(self) -> dict:
        out = {"rounds": dict(self.rounds), "emitted": dict(self.emitted)}
        if self.timed:
            out["seconds"] = {f"{r}_{ph}": round(v, 6) for (r, ph), v in self.seconds.items()}
        return out

