#!/usr/bin/env python3
"""SpecQuant round benchmark on one MI355X.

A step is one speculative round of the hot path (SpecQuant SS III-D) on a
synthetic Qwen2.5-shaped stack: k draft passes with the quantized draft copy
(dequant GEMVs, then a draft-token draw each), one verify pass with the FP16
parent (MFMA GEMMs at m = batch * (k + 1)), and the accept / resample step.
Rounds are replayed from a captured HIP graph; the timed region is K rounds
with the inputs resident in HBM.

Prints one JSON line: tokens/s (emitted tokens = accepted drafts + 1 per
sequence and round), the draft GEMV's achieved HBM bandwidth against the
MI355X peak, the CPU oracle timed on this host as a baseline, and the same
stack decoded directly with the FP16 parent (the paper's plain-decoding
comparison) with the speedup over it.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config 2]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E, GB/s
METRIC = "draft+verify tokens/s at Qwen2.5-7B shape (k=4); INT4/FP8 GEMV HBM TB/s vs peak"
CSRC = os.path.join(ROOT, "paper_2609_21704_amd", "csrc")
# the sources of each draft GEMV variant's kernels (a traffic profile is valid while they are unchanged)
GEMV_SOURCES = {"int4": ["gemv.hip"], "fp8": ["gemv.hip", "linear.hip"]}
FP8_CONFIG = 3         # the Qwen2.5-7B-shaped workload with the FP8 draft (m = 4)
COPY_BYTES = 1 << 30   # the plain copy that calibrates the HBM byte counters


def gemv_bytes(variant: str, m: int, n: int, k: int, out_bytes: int) -> float:
    """Algorithmic bytes of one draft GEMV launch: weights + activations + outputs."""
    w = n * k * 17 / 32 if variant == "int4" else n * k + 4 * n
    return w + 2 * m * k + m * n * out_bytes


def spin_cycles_per_ms() -> float:
    """Cycles of torch's spin kernel per millisecond on this device."""
    import torch

    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    torch.cuda._sleep(1 << 22)
    e1.record()
    torch.cuda.synchronize()
    return (1 << 22) / max(e0.elapsed_time(e1), 1e-3)


def measure_gemv(rnd, steps: int):
    """Average duration of a draft-GEMV launch: HIP events on the launching
    stream bracket the back-to-back GEMV launches of a whole draft pass (every
    layer's projections and the LM head), and the interval is divided by the
    launch count.  A spin kernel of about 40 ms runs first, so that every
    launch of the pass is queued before the GPU reaches it and no host-side
    launch latency lands inside the interval."""
    import torch

    cycles_per_ms = spin_cycles_per_ms()
    cfg, st = rnd.cfg, rnd.stack
    pass_bytes = 0.0
    n_launch = 0
    for l, name, n, k in st.mats:
        out_bytes = 4 if name == "lm_head" else 2
        pass_bytes += gemv_bytes(st.variant, cfg.draft_m, n, k, out_bytes)
        n_launch += 1
    tot_bytes, tot_s, launches = 0.0, 0.0, 0
    for i in range(steps):
        marks, calls = [], [0]

        def hook(start, marks=marks, calls=calls):
            j = calls[0]
            calls[0] += 1
            if j == 0 or j == 2 * n_launch - 1:  # before the first launch, after the last
                e = torch.cuda.Event(enable_timing=True)
                e.record()
                marks.append(e)

        torch.cuda._sleep(int(40 * cycles_per_ms))
        rnd.draft_step(i % cfg.k, on_gemv=hook)
        torch.cuda.synchronize()
        assert calls[0] == 2 * n_launch and len(marks) == 2
        tot_s += marks[0].elapsed_time(marks[1]) * 1e-3
        tot_bytes += pass_bytes
        launches += n_launch
    return tot_bytes, tot_s, launches


def measure_probe(rnd, steps: int, big_bytes: int = 4 << 30):
    """The measured read ceiling, with the library's streaming-read probe (one
    plain 16-byte-load read, nothing else):
      - `peak`: one read of a 4 GiB buffer (16 times the memory-side cache);
      - `same_launches`: one probe launch per draft-GEMV launch of a pass, each
        reading that launch's algorithmic bytes from a fresh place in the
        buffer, back to back and timed like the GEMVs -- what a pass of plain
        reads with the same launch sizes costs."""
    import torch

    from paper_2609_21704_amd import sq_probe_stream_read

    buf = torch.zeros(big_bytes, dtype=torch.uint8, device="cuda")
    sink = torch.empty(2048, dtype=torch.int32, device="cuda")
    for _ in range(2):
        sq_probe_stream_read(buf, sink=sink)
    torch.cuda.synchronize()
    best = float("inf")
    for _ in range(5):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        sq_probe_stream_read(buf, sink=sink)
        e1.record()
        torch.cuda.synchronize()
        best = min(best, e0.elapsed_time(e1) * 1e-3)
    peak = big_bytes / best / 1e9

    cfg, st = rnd.cfg, rnd.stack
    sizes = []
    for l, name, n, k in st.mats:
        b = gemv_bytes(st.variant, cfg.draft_m, n, k, 4 if name == "lm_head" else 2)
        sizes.append(max(16, int(b) // 16 * 16))
    cycles_per_ms = spin_cycles_per_ms()
    tot_s, tot_b, launches, off = 0.0, 0.0, 0, 0
    for _ in range(steps):
        torch.cuda.synchronize()
        torch.cuda._sleep(int(40 * cycles_per_ms))  # queue every launch before the GPU reaches the first
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for b in sizes:
            if off + b > big_bytes:
                off = 0
            sq_probe_stream_read(buf, b, off, sink=sink)
            off += (b + 4095) // 4096 * 4096
        e1.record()
        torch.cuda.synchronize()
        tot_s += e0.elapsed_time(e1) * 1e-3
        tot_b += sum(sizes)
        launches += len(sizes)
    del buf
    return {
        "kernel": "sq_probe_stream_read (plain 16-byte streaming read)",
        "peak_gbs": round(peak, 1),
        "peak_bytes": big_bytes,
        "same_launches_gbs": round(tot_b / tot_s / 1e9, 1),
        "same_launches_avg_us": round(tot_s / launches * 1e6, 3),
    }


def per_shape(cfg, rot_bytes: int = 3 << 30, iters: int = 40):
    """Back-to-back launches of each draft GEMV and verify GEMM shape of the
    workload, each over rotating copies of at least rot_bytes in all (so the
    memory-side cache cannot serve them), beside the read probe on the same
    bytes.  Weights are random bytes of the right layout (timing only)."""
    import torch

    import paper_2609_21704_amd as sq

    dev = torch.device("cuda")
    cpm = spin_cycles_per_ms()
    sink = torch.empty(2048, dtype=torch.int32, device=dev)

    def b2b(fn, copies):
        for i in range(3):
            fn(i % copies)
        torch.cuda.synchronize()
        torch.cuda._sleep(int(20 * cpm))
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for i in range(iters):
            fn(i % copies)
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) * 1e3 / iters

    shapes = [(name, n, k) for name, n, k in cfg.layer_matrices()]
    if cfg.lm_head:
        shapes.append(("lm_head", cfg.vocab, cfg.hidden))
    rows = []
    for name, n, k in shapes:
        m = cfg.draft_m
        if cfg.draft_variant == "int4":
            per = n * k // 2 + n * (k // 128) * 4
            copies = max(2, rot_bytes // per)
            codes = [torch.randint(0, 256, (n, k // 2), dtype=torch.uint8, device=dev) for _ in range(copies)]
            sc = [torch.full((n, k // 128), 0.01, dtype=torch.float16, device=dev) for _ in range(copies)]
            zz = [torch.full((n, k // 128), 8.0, dtype=torch.float16, device=dev) for _ in range(copies)]
            x = torch.randn((m, k), device=dev).half()
            y = torch.empty((m, n), device=dev, dtype=torch.float16)
            t_d = b2b(lambda i: sq.sq_qgemv_w4a16(x, codes[i], sc[i], zz[i], y=y), copies)
            b_d = gemv_bytes("int4", m, n, k, 2)
            del codes, sc, zz
        else:
            per = n * k + 4 * n
            copies = max(2, rot_bytes // per)
            codes = [torch.randint(0, 126, (n, k), dtype=torch.uint8, device=dev) for _ in range(copies)]
            sc = [torch.full((n,), 0.001, dtype=torch.float32, device=dev) for _ in range(copies)]
            x = torch.randn((m, k), device=dev).half()
            y = torch.empty((m, n), device=dev, dtype=torch.float16)
            t_d = b2b(lambda i: sq.sq_qgemv_w8a16(x, codes[i], sc[i], y=y), copies)
            b_d = gemv_bytes("fp8", m, n, k, 2)
            del codes, sc
        mv = cfg.verify_m
        copies = max(2, rot_bytes // (2 * n * k))
        w = [torch.empty((n, k), device=dev, dtype=torch.float16).normal_(0, 0.02) for _ in range(copies)]
        xv = torch.randn((mv, k), device=dev).half()
        yv = torch.empty((mv, n), device=dev, dtype=torch.float16)
        t_v = b2b(lambda i: sq.sq_verify_gemm_f16(xv, w[i], y=yv), copies)
        b_v = 2 * n * k + 2 * mv * k + 2 * mv * n
        del w
        buf = torch.zeros(rot_bytes, dtype=torch.uint8, device=dev)
        probe = {}
        for key, nb in (("draft", int(b_d) // 16 * 16), ("verify", int(b_v) // 16 * 16)):
            slots = max(2, rot_bytes // ((nb + 4095) // 4096 * 4096))
            step = (nb + 4095) // 4096 * 4096
            probe[key] = b2b(lambda i: sq.sq_probe_stream_read(buf, nb, (i % slots) * step, sink=sink), slots)
        del buf
        rows.append({"matrix": name, "n": n, "k": k,
                     "draft": {"m": m, "us": round(t_d, 2), "gbs": round(b_d / t_d / 1e3, 1),
                               "probe_us": round(probe["draft"], 2)},
                     "verify": {"m": mv, "us": round(t_v, 2), "gbs": round(b_v / t_v / 1e3, 1),
                                "probe_us": round(probe["verify"], 2)}})
    return rows


def sources_sha(variant: str) -> str:
    h = hashlib.sha256()
    for f in GEMV_SOURCES[variant]:
        h.update(open(os.path.join(CSRC, f), "rb").read())
    return h.hexdigest()


def traffic_from_profile(variant: str):
    """HBM bytes per draft-GEMV call from the committed rocprofv3 counter
    summary, if it was taken on the current kernel sources; else None."""
    path = os.path.join(ROOT, "profiles", f"gemv_{variant}_traffic.txt")
    if not os.path.exists(path):
        return None
    sha = sources_sha(variant)
    vals = {}
    for line in open(path):
        if "=" in line and not line.startswith("#"):
            key, val = line.split("=", 1)
            vals[key.strip()] = val.strip()
    if vals.get("gemv_source_sha256") != sha:
        return None
    try:
        return float(vals["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def cpu_baseline(rnd, tokens_per_round: float):
    """The fp64 CPU oracle on this host: layers 0 and L-1 plus the LM head, one
    full round of their work (k draft GEMVs, draws, verify GEMMs, accept),
    extrapolated to the whole stack."""
    import numpy as np
    import torch

    import oracle

    cfg, st, b = rnd.cfg, rnd.stack, rnd.buf
    T = rnd.temperature

    def bits(t):
        return t.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)

    layers = sorted({0, st.layers - 1})
    w16 = {}
    packs = {}
    for l in layers:
        for name, _, _ in cfg.layer_matrices():
            w16[(l, name)] = bits(st.w16[(l, name)])
    if cfg.lm_head:
        w16[(cfg.layers, "lm_head")] = bits(st.w16[(cfg.layers, "lm_head")])
    for key, w in w16.items():  # the oracle's own draft copy (not timed)
        packs[key] = oracle.quantize_int4_g128(w) if st.variant == "int4" else oracle.quantize_fp8_e4m3(w)
    xd = {key: bits(t) for key, t in b.xd.items() if key[2] == "lm_head" or key[1] in layers}
    xv = {key: bits(t) for key, t in b.xv.items() if key[1] == "lm_head" or key[0] in layers}

    def gemv(key, x):
        p = packs[key]
        return oracle.qgemv_w4a16(x, *p)[0] if st.variant == "int4" else oracle.qgemv_w8a16(x, *p)[0]

    eps = b.eps.cpu().numpy()
    u_d = b.u_draft.cpu().numpy().view(np.uint32)
    u_a = b.u_accept.cpu().numpy().view(np.uint32)
    t_layer_draft = t_lm_draft = t_sample = t_layer_verify = t_lm_verify = t_accept = 0.0
    B, k, V = cfg.batch, cfg.k, cfg.vocab
    draft_logits = np.zeros((k, B, V), np.float32) if cfg.lm_head else b.draft_logits.cpu().numpy()
    tokens = np.zeros((k, B), np.int32)
    for i in range(k):
        for l in layers:
            t0 = time.perf_counter()
            for name, _, _ in cfg.layer_matrices():
                gemv((l, name), xd[(i, l, name)])
            t_layer_draft += (time.perf_counter() - t0) / len(layers)
        if cfg.lm_head:
            t0 = time.perf_counter()
            draft_logits[i] = gemv((cfg.layers, "lm_head"), xd[(i, st.layers, "lm_head")]).astype(np.float32)
            t_lm_draft += time.perf_counter() - t0
        t0 = time.perf_counter()
        _, nxt, _, _ = oracle.spec_accept(None, draft_logits[i].reshape(B, 1, V), None,
                                          u_d[i].reshape(B, 1), T)
        t_sample += time.perf_counter() - t0
        tokens[i] = nxt
    for l in layers:
        t0 = time.perf_counter()
        for name, _, _ in cfg.layer_matrices():
            oracle.gemm_f16(xv[(l, name)], w16[(l, name)])
        t_layer_verify += (time.perf_counter() - t0) / len(layers)
    target = np.zeros((B, k + 1, V), np.float32)
    if cfg.lm_head:
        t0 = time.perf_counter()
        y = oracle.gemm_f16(xv[(st.layers, "lm_head")], w16[(cfg.layers, "lm_head")])[0]
        t_lm_verify = time.perf_counter() - t0
        target[:, k] = y.reshape(B, k + 1, V)[:, k]
    target[:, :k] = draft_logits.transpose(1, 0, 2) + eps
    t0 = time.perf_counter()
    oracle.spec_accept(draft_logits, target, tokens, u_a, T)
    t_accept = time.perf_counter() - t0
    # the draft terms already sum over the k draft steps
    round_s = (cfg.layers * t_layer_draft + t_lm_draft + t_sample
               + cfg.layers * t_layer_verify + t_lm_verify + t_accept)
    measured = (len(layers) * t_layer_draft + t_lm_draft + t_sample
                + len(layers) * t_layer_verify + t_lm_verify + t_accept)
    # one layer's draft GEMVs (one draft step) on one thread
    threads = oracle.num_threads()
    oracle.set_num_threads(1)
    t0 = time.perf_counter()
    for name, _, _ in cfg.layer_matrices():
        gemv((layers[0], name), xd[(0, layers[0], name)])
    t_single = time.perf_counter() - t0
    oracle.set_num_threads(threads)
    cpu_model = None
    try:  # lscpu's model name, else /proc/cpuinfo's
        import subprocess

        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=20).stdout
        cpu_model = next((l.split(":", 1)[1].strip() for l in out.splitlines() if l.startswith("Model name")), None)
    except (OSError, subprocess.SubprocessError):
        pass
    if not cpu_model:
        try:
            with open("/proc/cpuinfo") as f:
                cpu_model = next((l.split(":", 1)[1].strip() for l in f if l.startswith("model name")), None)
        except OSError:
            pass
    return {
        "value": round(tokens_per_round * cfg.batch / round_s, 4),
        "unit": "tokens/s",
        "cores": threads,
        "cpu_model": cpu_model,
        "single_thread_layer_draft_s": round(t_single, 3),
        "kind": "oracle",
        "sample": (f"layers {layers} of {cfg.layers} (4 projections each) and the LM head: one round of their "
                   f"draft GEMVs, draws, verify GEMMs and the accept step, timed in {measured:.1f} s and "
                   f"extrapolated to {cfg.layers} layers ({round_s:.1f} s per round)"),
    }


def expected_tokens(rnd, ud, ua, rounds, n_hist):
    """The expected tokens per round of each timed round from its own
    distributions: with draft rows q_j and parent rows p_j fixed in a round,
    position j is accepted with probability beta_j = sum_x min(p_j(x), q_j(x))
    independently of the others, so E[n + 1] = 1 + sum_{i=1..k} prod_{j<i} beta_j.
    Each round is run again eagerly with its uniforms (its n_accepted must equal
    the timed replay's), and its accept step once more with q_out / p_out."""
    import torch

    from paper_2609_21704_amd import sq_spec_accept

    cfg, b = rnd.cfg, rnd.buf
    B, k, V = cfg.batch, cfg.k, cfg.vocab
    q = torch.empty((k, B, V), dtype=torch.float32, device=b.n_accepted.device)
    p = torch.empty((B, k + 1, V), dtype=torch.float32, device=b.n_accepted.device)
    per_round = []
    for r in rounds:
        rnd.set_uniforms(ud[r], ua[r])
        rnd.run()
        n2, _ = sq_spec_accept(b.draft_logits, b.target_logits, b.draft_tokens, b.u_accept, rnd.temperature,
                               q_out=q, p_out=p)
        if not torch.equal(n2, n_hist[r]) or not torch.equal(b.n_accepted, n_hist[r]):
            raise RuntimeError(f"round {r} did not reproduce its timed replay")
        beta = torch.minimum(p[:, :k].double(), q.permute(1, 0, 2).double()).sum(dim=2)   # [B][k]
        e = 1.0 + torch.cumprod(beta, dim=1).sum(dim=1)                                   # [B]
        per_round.append(e.mean().item())
    return sum(per_round) / len(per_round), beta.mean(dim=0).tolist()


def measure_fp8(steps: int, dev):
    """The W8A16 draft GEMVs at m = 4 over the Qwen2.5-7B FP8 workload's shapes
    (28 layers' projections and the LM head), timed like the INT4 ones."""
    import torch

    from paper_2609_21704_amd.configs import CONFIGS
    from paper_2609_21704_amd.rounds import Round, Stack

    cfg = CONFIGS[FP8_CONFIG]
    stack = Stack(cfg, dev, keep_f16=False)
    rnd = Round(stack, temperature=1.0)
    for i in range(cfg.k):  # one untimed pass of every draft step first
        rnd.draft_step(i)
    torch.cuda.synchronize()
    gbytes, gsec, glaunch = measure_gemv(rnd, steps)
    achieved = gbytes / gsec / 1e9
    out = {
        "kernel": f"draft GEMV (W8A16, m={cfg.draft_m})",
        "workload": cfg.describe(),
        "bound": "hbm",
        "achieved": round(achieved, 1),
        "peak": HBM_PEAK_GBS,
        "unit": "GB/s",
        "frac": round(achieved / HBM_PEAK_GBS, 4),
        "traffic": traffic_from_profile("fp8"),
        "launches_timed": glaunch,
        "avg_launch_us": round(gsec / glaunch * 1e6, 3),
        "algorithmic_bytes_per_launch": round(gbytes / glaunch, 1),
    }
    del rnd, stack
    torch.cuda.empty_cache()
    return out


def measure_direct(stack, temperature: float, steps: int, warmup: int):
    """Direct parent inference (SS III-D.5), the paper's plain-decoding
    baseline: one token per sequence per step from the FP16 parent alone,
    timed over graph replays like the rounds."""
    import torch

    from paper_2609_21704_amd import synth
    from paper_2609_21704_amd.rounds import DirectDecode

    cfg = stack.cfg
    dd = DirectDecode(stack, temperature=temperature)
    dd.u.copy_(synth.uniform_u24((cfg.batch, 1), synth.stream_seed(cfg.seed, 99), dd.u.device))
    dd.capture()
    for _ in range(warmup):
        dd.replay()
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        dd.replay()
    e1.record()
    torch.cuda.synchronize()
    sec = e0.elapsed_time(e1) * 1e-3
    return {
        "tokens_per_s": round(cfg.batch * steps / sec, 3),
        "ms_per_token": round(sec / steps * 1e3, 4),
        "steps": steps,
        "what": "plain FP16 decoding at m = batch: every FP16 matrix streamed once per token, then a draw",
    }


DECODER_CONTEXT = 1024   # prompt tokens in both caches when the timed decoder rounds start
DECODER_CAPACITY = 2048  # cache positions per sequence


def measure_decoder(stack, temperature: float, steps: int, warmup: int, chains: int = 1):
    """The same rounds through full decoder layers with key/value caches
    (embedding, RMSNorm, q|k|v + bias, RoPE, causal GQA attention over the
    cache, SiLU-gated product, residuals; the matrices are the stack's): a
    synthetic prompt of DECODER_CONTEXT tokens is prefilled, then graph
    replays of whole rounds are timed; each round commits its tokens and rolls
    both caches back to the accepted prefix.  The attention calls of one eager
    round are timed with events for their roofline (HBM: 512 bytes per cached
    position and kv head, plus the queries and outputs).  With chains > 1 each
    sequence drafts that many independent chains, verified in one pass and
    accepted over their prefix tree."""
    import numpy as np
    import torch

    from paper_2609_21704_amd import decoder as dec
    from paper_2609_21704_amd import synth

    cfg = stack.cfg
    B, k = cfg.batch, cfg.k
    w = dec.DecoderWeights(cfg, stack.device, stack=stack)
    sd = dec.SpecDecoder(w, capacity=DECODER_CAPACITY, temperature=temperature, chains=chains)
    sd.prefill(dec.synthetic_prompt(cfg, B, DECODER_CONTEXT, stack.device))
    total = 2 + warmup + steps  # round 0: eager attention timing, round 1: the eager run of capture
    ud = synth.uniform_u24((total, k, B * chains), synth.stream_seed(cfg.seed, 120, chains), stack.device)
    ua = synth.uniform_u24((total, B, chains * k + 1), synth.stream_seed(cfg.seed, 121, chains), stack.device)
    n_hist = torch.zeros((total, B), dtype=torch.int32, device=stack.device)

    # round 0, eager: events around every attention call (positions are fixed until the commit)
    calls = []

    def hook(start, rps, offset):
        ev = torch.cuda.Event(enable_timing=True)
        ev.record()
        if start:
            calls.append([ev, None, rps, offset])
        else:
            calls[-1][1] = ev

    pos = sd.pos_base.cpu().numpy().astype(np.int64)
    sd.attn_hook = hook
    sd.set_uniforms(ud[0], ua[0])
    sd.run()
    sd.attn_hook = None
    torch.cuda.synchronize()
    n_hist[0].copy_(sd.n_accepted)
    att_bytes, att_sec = 0.0, 0.0
    for e0, e1, rps, offset in calls:
        att_sec += e0.elapsed_time(e1) * 1e-3
        last = pos + offset + rps - 1
        att_bytes += float(((last + 1) * 512 * cfg.kv_heads).sum()) + 2 * B * chains * rps * cfg.q_dim * 2

    sd.set_uniforms(ud[1], ua[1])
    sd.capture()
    n_hist[1].copy_(sd.n_accepted)

    def one(r):
        sd.set_uniforms(ud[r], ua[r])
        sd.replay()
        n_hist[r].copy_(sd.n_accepted)

    for r in range(2, 2 + warmup):
        one(r)
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    pos0 = sd.pos_base[::chains].clone()
    e0.record()
    for r in range(2 + warmup, total):
        one(r)
    e1.record()
    torch.cuda.synchronize()
    sec = e0.elapsed_time(e1) * 1e-3
    n_acc = n_hist[2 + warmup:].cpu().numpy().astype(np.int64)
    tokens = int((n_acc + 1).sum())
    assert int((sd.pos_base[::chains] - pos0).sum().item()) == tokens, "positions moved by the emitted tokens"
    assert sd.status.item() == 0, "device status flags raised"
    achieved = att_bytes / att_sec / 1e9
    return {
        "tokens_per_s": round(tokens / sec, 3),
        "ms_per_round": round(sec / steps * 1e3, 4),
        "rounds": steps,
        "tokens_per_round": round(tokens / (steps * B), 4),
        "acceptance_rate": round(float(n_acc.sum()) / (steps * B * k), 4),
        "chains": chains,
        "context_at_start": DECODER_CONTEXT,
        "cache_capacity": DECODER_CAPACITY,
        "what": "rounds through Qwen2.5-7B-shaped decoder layers (RMSNorm, q|k|v + bias, RoPE, GQA attention "
                "over the KV cache, SiLU-gated MLP, residuals; random weights), the caches rolled back to the "
                "accepted prefix each round",
        "roofline_attention": {
            "kernel": "attention over the cache (chunk partials + ordered merge), one eager round",
            "bound": "hbm",
            "achieved": round(achieved, 1),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4),
            "calls": len(calls),
            "avg_call_us": round(att_sec / len(calls) * 1e6, 3),
            "algorithmic_bytes_per_call": round(att_bytes / len(calls), 1),
        },
    }


ROUTED_REQUESTS = 16  # text requests of the routed measurement
ROUTED_NEW = 32       # tokens generated per request


def measure_routed(stack, temperature: float):
    """The execution pipeline end to end: ROUTED_REQUESTS synthetic text
    requests are scored by the router and served by speculative decoding with
    the INT4 or FP8 draft or by direct FP16 decoding (one parent, both drafts
    resident), four sequences per batch, ROUTED_NEW tokens each; then the same
    requests all decoded directly.  Wall time covers tokenisation, ragged
    prefill of both caches, graph replays of the rounds and the host's checks
    between rounds; the prefill and round phases are also given apart."""
    import time

    import torch

    from paper_2609_21704_amd import decoder as dec
    from paper_2609_21704_amd import synth
    from paper_2609_21704_amd.engine import Engine
    from paper_2609_21704_amd.router import ROUTES

    cfg = stack.cfg
    w = dec.DecoderWeights(cfg, stack.device, stack=stack)
    eng = Engine(cfg, stack.device, k=cfg.k, batch=4, capacity=1024, temperature=temperature, parent=w,
                 timed=True)
    texts = synth.prompt_texts(ROUTED_REQUESTS, cfg.seed)
    # untimed: every route once (library workspace, graph capture)
    eng.generate([texts[0]] * 3, 4, routes=list(ROUTES))

    def run(routes):
        before = eng.stats()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        res = eng.generate(texts, ROUTED_NEW, routes=routes)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        after = eng.stats()
        sec = {key: after["seconds"][key] - before["seconds"][key] for key in after["seconds"]}
        rounds = {r: after["rounds"][r] - before["rounds"][r] for r in ROUTES}
        tokens = sum(len(x.tokens) for x in res)
        pre = sum(v for key, v in sec.items() if key.endswith("prefill"))
        dec_s = sum(v for key, v in sec.items() if key.endswith("rounds"))
        per_route = {}
        for r in ROUTES:
            n = sum(x.served_by == r for x in res)
            if n:
                per_route[r] = {"requests": n, "rounds": rounds[r],
                                "decode_tokens_per_s": round(n * ROUTED_NEW / sec[f"{r}_rounds"], 2),
                                "prefill_s": round(sec[f"{r}_prefill"], 4)}
        return res, {"tokens_per_s": round(tokens / wall, 2), "wall_s": round(wall, 4), "prefill_s": round(pre, 4),
                     "rounds_s": round(dec_s, 4), "decode_tokens_per_s": round(tokens / dec_s, 2),
                     "per_route": per_route}

    res, routed = run(None)
    _, direct = run(["f16"] * len(texts))
    del eng, w
    torch.cuda.empty_cache()
    mix = {r: sum(x.route == r for x in res) for r in ROUTES}
    return {
        "what": "synthetic text requests routed by prompt complexity (INT4 / FP8 speculative, FP16 direct) through "
                "the 7B-shaped decoder, against the same requests all decoded directly",
        "requests": len(texts),
        "new_tokens_each": ROUTED_NEW,
        "prompt_tokens": [x.prompt_tokens for x in res],
        "mix": mix,
        "temperature": temperature,
        "routed": routed,
        "all_direct": direct,
        "speedup_vs_all_direct": round(routed["tokens_per_s"] / direct["tokens_per_s"], 3),
        "decode_speedup_vs_all_direct": round(routed["decode_tokens_per_s"] / direct["decode_tokens_per_s"], 3),
    }


def measure_attention_long(dev, context: int = 8192, batch: int = 4, rows: int = 9, iters: int = 20):
    """The attention call alone at a bandwidth-sized shape: 4 sequences of
    8192 cached positions with Qwen2.5-7B heads (28 q / 4 kv), 9 rows per
    sequence (a k = 8 verification block), over rotating caches (so that no
    cache level holds them between calls); HBM roofline of 512 bytes per
    cached position and kv head plus the queries and outputs."""
    import torch

    import paper_2609_21704_amd as sq

    hq, hkv = 28, 4
    copies = 4
    kc = [torch.randn((batch, hkv, context, 128), device=dev).half() for _ in range(copies)]
    vc = [torch.randn((batch, hkv, 128, context), device=dev).half() for _ in range(copies)]
    q = torch.randn((batch * rows, hq, 128), device=dev).half()
    out = torch.empty_like(q)
    pb = torch.full((batch,), context - rows, dtype=torch.int32, device=dev)
    for i in range(3):
        sq.sq_attention_f16(q, kc[i % copies], vc[i % copies], pb, 0, rows, out=out)
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record()
    for i in range(iters):
        sq.sq_attention_f16(q, kc[i % copies], vc[i % copies], pb, 0, rows, out=out)
    e1.record()
    torch.cuda.synchronize()
    sec = e0.elapsed_time(e1) * 1e-3 / iters
    nbytes = batch * hkv * context * 512 + 2 * batch * rows * hq * 128 * 2
    del kc, vc
    return {
        "kernel": "attention over the cache (chunk partials + ordered merge)",
        "shape": f"{batch} sequences x {context} cached positions, 28 q / 4 kv heads of 128, {rows} rows each",
        "bound": "hbm",
        "achieved": round(nbytes / sec / 1e9, 1),
        "peak": HBM_PEAK_GBS,
        "unit": "GB/s",
        "frac": round(nbytes / sec / 1e9 / HBM_PEAK_GBS, 4),
        "avg_call_us": round(sec * 1e6, 3),
        "algorithmic_bytes_per_call": nbytes,
    }


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200, help="timed rounds")
    ap.add_argument("--warmup", type=int, default=20, help="untimed rounds")
    ap.add_argument("--config", type=int, default=2, help="workload index (2 = Qwen2.5-7B-shaped, INT4, k=4)")
    ap.add_argument("--temperature", type=float, default=1.0)
    ap.add_argument("--gemv-steps", type=int, default=2, help="draft passes timed per launch for the roofline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--per-shape", action="store_true",
                    help="instead of rounds: back-to-back launches of each draft GEMV and verify GEMM shape of "
                         "the workload, beside plain reads of the same bytes; one JSON line")
    ap.add_argument("--profile-only", action="store_true",
                    help="for rocprofv3 counter runs: one eager round, then a plain copy of COPY_BYTES bytes "
                         "(the counter calibration); prints nothing")
    ap.add_argument("--profile-draft", action="store_true",
                    help="for rocprofv3 counter runs: one eager pass of every draft step (GEMVs and draws), then "
                         "the plain copy; prints nothing")
    ap.add_argument("--no-fp8", action="store_true", help="skip the FP8 draft GEMV roofline block")
    ap.add_argument("--no-decoder", action="store_true", help="skip the rounds through full decoder layers")
    ap.add_argument("--no-pipeline", action="store_true", help="skip the routed requests through the pipeline")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py measures one GPU only: the SpecQuant hot path is built and timed on a single MI355X; "
              f"its sharding over several GPUs is a design, not code (requested --gpus {args.gpus}).",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2609_21704_amd.configs import CONFIGS
    from paper_2609_21704_amd.rounds import Round, Stack, round_uniforms

    cfg = CONFIGS[args.config]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.per_shape:
        print(json.dumps({"workload": cfg.describe(), "per_shape": per_shape(cfg)}), flush=True)
        return
    stack = Stack(cfg, dev, keep_f16=not args.profile_draft)
    rnd = Round(stack, temperature=args.temperature)
    if args.profile_only or args.profile_draft:
        ud, ua = round_uniforms(cfg, 1, dev)
        rnd.set_uniforms(ud[0], ua[0])
        if args.profile_draft:
            for i in range(cfg.k):
                rnd.draft_step(i)
        else:
            rnd.run()
        src = torch.empty(COPY_BYTES, dtype=torch.uint8, device=dev).fill_(1)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        torch.bitwise_not(src, out=dst)  # reads and writes each byte once: the last dispatch of the run
        torch.cuda.synchronize()
        return
    total = args.warmup + args.steps
    ud, ua = round_uniforms(cfg, total, dev)
    n_hist = torch.zeros((total, cfg.batch), dtype=torch.int32, device=dev)
    rnd.set_uniforms(ud[0], ua[0])
    rnd.capture()  # one eager round first (library workspace), then the graph

    def one(r):
        rnd.set_uniforms(ud[r], ua[r])
        rnd.replay()
        n_hist[r].copy_(rnd.buf.n_accepted)

    for r in range(args.warmup):
        one(r)
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    marks = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps - 1)]
    t0 = time.perf_counter()
    e0.record()
    for i, r in enumerate(range(args.warmup, total)):
        if i:
            marks[i - 1].record()
        one(r)
    e1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    elapsed = e0.elapsed_time(e1) * 1e-3
    edges = [e0, *marks, e1]
    round_ms = np.array([edges[i].elapsed_time(edges[i + 1]) for i in range(args.steps)])
    n_acc = n_hist[args.warmup:].cpu().numpy().astype(np.int64)
    tokens = int((n_acc + 1).sum())
    tokens_per_round = tokens / (args.steps * cfg.batch)

    expected, beta = expected_tokens(rnd, ud, ua, range(args.warmup, total), n_hist)
    direct = measure_direct(stack, args.temperature, args.steps, args.warmup)
    gbytes, gsec, glaunch = measure_gemv(rnd, args.gemv_steps)
    achieved = gbytes / gsec / 1e9
    traffic = traffic_from_profile(stack.variant)
    probe = measure_probe(rnd, args.gemv_steps)

    out = {
        "metric": METRIC,
        "value": round(tokens / elapsed, 3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(elapsed / args.steps * 1e3, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16",
        "data": "synthetic (seeded random weights and activations; no trained weights or datasets)",
        "config": {
            "workload": cfg.describe(),
            "draft_variant": stack.variant,
            "k": cfg.k,
            "batch": cfg.batch,
            "draft_m": cfg.draft_m,
            "verify_m": cfg.verify_m,
            "vocab": cfg.vocab,
            "temperature": args.temperature,
            "graph": True,
        },
        "rounds_per_s": round(args.steps / elapsed, 3),
        "round_ms": {"median": round(float(np.median(round_ms)), 4),
                     "p10": round(float(np.percentile(round_ms, 10)), 4),
                     "p90": round(float(np.percentile(round_ms, 90)), 4)},
        "tokens_per_round": round(tokens_per_round, 4),
        "expected_tokens_per_round": round(expected, 4),
        "acceptance_beta": [round(x, 4) for x in beta],
        "acceptance_rate": round(float(n_acc.sum()) / (args.steps * cfg.batch * cfg.k), 4),
        "round_bytes": cfg.round_bytes(),
        "stack_gbs": round(cfg.round_bytes() * args.steps / elapsed / 1e9, 1),
        "wall_s": round(wall, 4),
        "direct_parent": direct,
        "speedup_vs_direct": round(tokens / elapsed / direct["tokens_per_s"], 3),
        "roofline": {
            "kernel": f"draft GEMV ({'W4A16' if stack.variant == 'int4' else 'W8A16'}, m={cfg.draft_m})",
            "bound": "hbm",
            "achieved": round(achieved, 1),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4),
            "traffic": traffic,
            "launches_timed": glaunch,
            "avg_launch_us": round(gsec / glaunch * 1e6, 3),
            "algorithmic_bytes_per_launch": round(gbytes / glaunch, 1),
            "measured_peak": probe["peak_gbs"],
            "frac_of_measured_peak": round(achieved / probe["peak_gbs"], 4),
            "probe": probe,
            "frac_of_probe_same_launches": round(achieved / probe["same_launches_gbs"], 4),
        },
    }
    if not args.no_decoder:
        out["decoder"] = measure_decoder(stack, args.temperature, args.steps, args.warmup)
        out["decoder"]["roofline_attention_long"] = measure_attention_long(dev)
        out["decoder_chains"] = measure_decoder(stack, args.temperature, args.steps, args.warmup, chains=4)
        del out["decoder_chains"]["roofline_attention"]
        if not args.no_pipeline:
            out["pipeline"] = measure_routed(stack, args.temperature)
    if not args.no_fp8 and cfg.draft_variant == "int4":
        out["roofline_fp8"] = measure_fp8(args.gemv_steps, dev)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(rnd, tokens_per_round)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
