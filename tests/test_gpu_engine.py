"""GPU tests of the execution pipeline (SS III-D): direct parent decoding
(SS III-D.5), ragged prompts prefilled together, the engine's three routes
(INT4 and FP8 speculative decoding, FP16 direct; SS III-B) over one shared
parent (SS III-A), and the placement fallback (SS III-C).

Greedy decoding is checked teacher-forced against the fp64 oracle: the oracle
runs each sequence's prompt and emitted tokens through the parent, and every
emitted token must be the oracle's argmax up to the logits tolerance of the
decoder tests (the GPU's logits lie within 1e-2 of the rms of the oracle's,
so a token within 2e-2 rms of the top is a legitimate argmax of a near tie).
Speculative decoding emits the parent's greedy tokens, so the three routes
must agree token for token up to the first such near tie."""
import numpy as np
import pytest
import torch

from oracle import decoder as od

import paper_2609_21704_amd as sq
from paper_2609_21704_amd import decoder as dec
from paper_2609_21704_amd import synth
from paper_2609_21704_amd.configs import CONFIGS
from paper_2609_21704_amd.engine import Engine, cache_bytes, placement, weight_bytes
from paper_2609_21704_amd.router import Router

pytestmark = pytest.mark.gpu
DEV = "cuda"
TIE = 2e-2  # of the rms of a row of logits


def parent_model(w):
    cfg = w.cfg
    dims = od.Dims(w.layers, cfg.hidden, cfg.intermediate, cfg.q_heads, cfg.kv_heads, cfg.vocab,
                   eps=dec.EPS, theta=dec.THETA)
    return dims, od.Model(dims, w.params(), "f16")


def oracle_logits(dims, model, seq):
    """Parent logits at every position of one sequence (fp64, teacher-forced)."""
    cache = od.Cache(dims, 1, ((len(seq) + 63) // 64) * 64)
    return od.forward(model, cache, np.asarray(seq)[None, :], np.arange(len(seq))[None, :])[0]


def check_greedy(dims, model, prompt, emitted, what):
    """Every emitted token is the oracle parent's argmax up to a near tie;
    returns the oracle's top-2 gaps / rms per emitted token."""
    seq = list(prompt) + list(emitted)
    L = oracle_logits(dims, model, seq[:-1])[len(prompt) - 1:]
    gaps = []
    for j, t in enumerate(emitted):
        row = L[j]
        rms = np.sqrt(np.mean(row * row))
        assert row.max() - row[t] <= TIE * rms, f"{what}: token {j} ({t}) is {(row.max() - row[t]) / rms:.3e} rms " \
                                               f"below the argmax {int(np.argmax(row))}"
        top2 = np.sort(row)[-2:]
        gaps.append((top2[1] - top2[0]) / rms)
    return gaps


def agree_until_near_tie(a, b, gaps, what):
    for j, (x, y) in enumerate(zip(a, b)):
        if x != y:
            assert gaps[j] <= 2 * TIE, f"{what}: token {j} differs ({x} vs {y}) with a top-2 gap of {gaps[j]:.3e}"
            return j
    return len(a)


def ragged_prompts(cfg, lengths, seed):
    return [synth.tokens((n,), cfg.vocab, synth.stream_seed(seed, i), "cpu").tolist() for i, n in enumerate(lengths)]


# ----------------------------------------------------------- direct decoding
@pytest.mark.parametrize("ci,layers,lengths,steps", [(0, 1, [5, 17, 30], 12), (1, 2, [9, 2], 6)])
def test_direct_decoder_matches_oracle(ci, layers, lengths, steps):
    cfg = CONFIGS[ci]
    print(f"\n[direct] config {ci} layers {layers} prompts {lengths}", flush=True)
    w = dec.DecoderWeights(cfg, DEV, layers=layers, variant="int4")
    B = len(lengths)
    dd = dec.DirectDecoder(w, batch=B, capacity=128, temperature=0.0)
    prompts = ragged_prompts(cfg, lengths, 7 + ci)
    pad = torch.zeros((B, max(lengths)), dtype=torch.int32)
    for b, p in enumerate(prompts):
        pad[b, :len(p)] = torch.tensor(p)
        pad[b, len(p):] = 3  # padding, never attended to
    dd.prefill(pad, lengths=lengths)
    assert dd.pos_base.cpu().tolist() == [n - 1 for n in lengths]
    dims, model = parent_model(w)
    logits = []
    for s in range(steps):
        dd.set_uniforms(torch.zeros((B, 1), dtype=torch.int32, device=DEV))
        dd.run()
        logits.append(dd.logits.cpu().numpy().copy())
    torch.cuda.synchronize()
    assert dd.status.item() == 0
    out, out_len = dd.out_tokens.cpu().numpy(), dd.out_len.cpu().numpy()
    assert (out_len == steps).all()
    assert dd.pos_base.cpu().tolist() == [n - 1 + steps for n in lengths]
    for b in range(B):
        em = out[b, :steps].tolist()
        g = np.stack([l[b] for l in logits])
        assert np.array_equal(np.argmax(g, axis=1), em)  # the kernel's own argmax
        seq = prompts[b] + em
        ref = oracle_logits(dims, model, seq[:-1])[lengths[b] - 1:]
        rms = np.sqrt(np.mean(ref * ref, axis=1, keepdims=True))
        d = np.abs(g - ref) / rms
        assert d.max() <= 1e-2 and d.mean() <= 2e-3, f"sequence {b}: logits max {d.max():.2e} mean {d.mean():.2e}"
        check_greedy(dims, model, prompts[b], em, f"sequence {b}")


def test_direct_decoder_graph_replays():
    cfg = CONFIGS[0]
    w = dec.DecoderWeights(cfg, DEV, layers=1, variant="int4")
    prompts = ragged_prompts(cfg, [6, 11], 3)
    pad = torch.zeros((2, 11), dtype=torch.int32)
    for b, p in enumerate(prompts):
        pad[b, :len(p)] = torch.tensor(p)
    u = synth.uniform_u24((8, 2, 1), 44, DEV)
    outs = []
    for graph in (False, True):
        dd = dec.DirectDecoder(w, batch=2, capacity=64, temperature=1.0)
        dd.prefill(pad, lengths=[6, 11])
        for s in range(8):
            dd.set_uniforms(u[s])
            if not graph:
                dd.run()
            elif dd.graph is None:
                dd.capture()
            else:
                dd.replay()
            torch.cuda.synchronize()
        outs.append(dd.out_tokens[:, :8].cpu())
    assert torch.equal(outs[0], outs[1])


# ------------------------------------------------------------------ engine
@pytest.mark.parametrize("ci,layers,k,batch,chains,lengths,max_new", [
    (0, 1, 3, 2, 1, [4, 19, 33, 8, 12], 14),
    (0, 1, 4, 1, 2, [10, 25], 11),
    (1, 2, 4, 2, 1, [7, 16, 3], 9),
])
def test_engine_routes_decode_the_parents_greedy_tokens(ci, layers, k, batch, chains, lengths, max_new):
    cfg = CONFIGS[ci]
    print(f"\n[engine] config {ci} layers {layers} k {k} batch {batch} chains {chains} prompts {lengths}", flush=True)
    eng = Engine(cfg, DEV, layers=layers, k=k, batch=batch, capacity=128, temperature=0.0, chains=chains)
    assert eng.plan["resident"] == ["f16", "int4", "fp8"]
    prompts = ragged_prompts(cfg, lengths, 11 + ci)
    n = len(prompts)
    results = {}
    for route in ("int4", "fp8", "f16"):
        res = eng.generate(prompts, max_new, routes=[route] * n)
        assert all(r.route == route and r.served_by == route and len(r.tokens) == max_new for r in res)
        results[route] = [r.tokens for r in res]
    dims, model = parent_model(eng.weights["f16"])
    agreed = []
    for i, p in enumerate(prompts):
        gaps = check_greedy(dims, model, p, results["f16"][i], f"f16 prompt {i}")
        for route in ("int4", "fp8"):
            check_greedy(dims, model, p, results[route][i], f"{route} prompt {i}")
            agreed.append(agree_until_near_tie(results[route][i], results["f16"][i], gaps, f"{route} prompt {i}"))
    assert sum(agreed) >= len(agreed) * max_new // 2  # near ties are rare
    st = eng.stats()
    assert st["emitted"] == {r: n * max_new for r in ("int4", "fp8", "f16")}
    # speculation emits several tokens per round
    assert st["rounds"]["int4"] < st["rounds"]["f16"]
    print(f"[engine] agreement {agreed}, rounds {st['rounds']}", flush=True)


def test_engine_text_requests_follow_the_router():
    cfg = CONFIGS[0]
    texts = synth.prompt_texts(7, 21)
    router = Router().calibrate(synth.prompt_texts(300, 22))
    eng = Engine(cfg, DEV, layers=1, k=3, batch=2, capacity=512, temperature=1.0, router=router, seed=5)
    res = eng.generate(texts, 6)
    for t, r in zip(texts, res):
        assert r.route == router.route(t) == r.served_by
        assert r.prompt_tokens == len(eng.tokenize(t))
        assert len(r.tokens) == 6 and all(0 <= x < cfg.vocab for x in r.tokens)
    assert len({r.route for r in res}) >= 2
    # a second engine with the same seed draws the same tokens
    eng2 = Engine(cfg, DEV, layers=1, k=3, batch=2, capacity=512, temperature=1.0, router=router, seed=5)
    assert [r.tokens for r in eng2.generate(texts, 6)] == [r.tokens for r in res]


def test_engine_placement_falls_back_when_a_draft_does_not_fit():
    cfg = CONFIGS[0]
    L, B, cap, k = 1, 2, 128, 3
    w = weight_bytes(cfg, L)
    c1 = cache_bytes(cfg, L, B, cap)
    free = (w["f16"] + c1 + w["int4"] + 2 * c1) / 0.9 + 1000
    assert placement(cfg, free, B, cap, k, L)["resident"] == ["f16", "int4"]
    eng = Engine(cfg, DEV, layers=L, k=k, batch=B, capacity=cap, temperature=0.0, free_bytes=free)
    assert set(eng.weights) == {"f16", "int4"}
    prompts = ragged_prompts(cfg, [5, 9, 14], 31)
    res = eng.generate(prompts, 5, routes=["fp8", "int4", "f16"])
    assert [r.served_by for r in res] == ["int4", "int4", "f16"]
    # only the parent fits: no draft copy is built and every request decodes directly
    free = (w["f16"] + c1) / 0.9 + 1000
    eng = Engine(cfg, DEV, layers=L, k=k, batch=B, capacity=cap, temperature=0.0, free_bytes=free)
    assert set(eng.weights) == {"f16"} and eng.weights["f16"].stack.draft == {}
    res = eng.generate(prompts, 5, routes=["fp8", "int4", "f16"])
    assert [r.served_by for r in res] == ["f16"] * 3


def test_variants_share_one_parent_and_weight_bytes():
    cfg = CONFIGS[1]
    L = 2
    eng = Engine(cfg, DEV, layers=L, k=4, batch=1, capacity=64)
    p, i4, f8 = eng.weights["f16"], eng.weights["int4"], eng.weights["fp8"]
    assert i4 is p and f8.stack.w16 is p.stack.w16 and f8.embed is p.embed
    for key, w16 in p.stack.w16.items():
        codes, scales = f8.stack.draft[key]
        c2, s2 = sq.sq_quantize_fp8_e4m3(w16)
        assert torch.equal(codes, c2) and torch.equal(scales, s2)
    wb = weight_bytes(cfg, L)
    nbytes = lambda ts: sum(t.numel() * t.element_size() for t in ts)  # noqa: E731
    parent = list(p.stack.w16.values()) + [p.embed, p.final_norm] + p.in_norm + p.post_norm + p.qkv_bias
    assert nbytes(parent) == wb["f16"]
    assert nbytes([t for v in i4.stack.draft.values() for t in v]) == wb["int4"]
    assert nbytes([t for v in f8.stack.draft.values() for t in v]) == wb["fp8"]


def test_engine_rejects_bad_requests():
    cfg = CONFIGS[0]
    eng = Engine(cfg, DEV, layers=1, k=3, batch=2, capacity=64)
    with pytest.raises(ValueError):
        eng.generate([[1]], 4)                     # a one-token prompt
    with pytest.raises(ValueError):
        eng.generate([[1, 2, 3]], 60)              # past the cache
    with pytest.raises(ValueError):
        eng.generate([[1, cfg.vocab]], 4)          # a token outside the vocabulary
    with pytest.raises(ValueError):
        eng.generate([[1, 2]], 4, routes=["q2"])   # an unknown route
