"""Pins of the decoder-step oracle (the layer around the projections of the
draft pass, SS III-D.2, and of the verification pass, SS III-D.3, for the
Qwen2.5 family the paper evaluates, SS IV) and of the speculative round with
its key/value cache (restart after a rejection, SS III-D.4).

Each operation is checked against something other than itself: worked
examples and closed forms (RMSNorm of (3, 4); a two-key attention whose
weights are exactly 1/4 and 3/4; rotation by exactly 1 radian), an independent
formulation (RoPE as complex multiplication, SiLU through scipy's logistic),
invariants (norm preservation, relative-position dependence, causality,
grouped-query head mapping), and, for the cache and the round, two identities
that hold for any correct implementation: decoding one token at a time through
the cache gives the logits of one pass over the whole sequence, and greedy
speculative decoding emits exactly the parent's greedy decode whatever the
draft proposes."""
import math

import numpy as np
import pytest
from scipy import special

import oracle
from oracle import decoder as od

RNG = np.random.default_rng(7)
D = od.HEAD_DIM


# ------------------------------------------------------------------ rmsnorm
def test_rmsnorm_worked_example_and_closed_forms():
    # (3, 4): mean square 12.5, rms 5 / sqrt(2)
    y = oracle.rmsnorm(np.array([[3.0, 4.0]]), np.ones(2), 0.0)
    assert np.allclose(y, [[3 * math.sqrt(2) / 5, 4 * math.sqrt(2) / 5]], rtol=1e-15, atol=0)
    # constant row c: c / sqrt(c^2 + eps) * w (eps inside the root)
    w = np.array([0.5, 2.0, -1.0])
    y = oracle.rmsnorm(np.full((1, 3), 0.01), w, 1e-4)
    assert np.allclose(y, 0.01 / math.sqrt(1e-4 + 1e-4) * w, rtol=1e-14, atol=0)
    # eps = 0: unit rms, and scale invariance up to the sign
    h = RNG.normal(0, 3, (4, 257))
    y = oracle.rmsnorm(h, np.ones(257), 0.0)
    assert np.allclose(np.sqrt(np.mean(y * y, axis=1)), 1.0, rtol=1e-14)
    assert np.allclose(oracle.rmsnorm(-7.5 * h, np.ones(257), 0.0), -y, rtol=1e-13, atol=1e-15)
    # the weight scales each column
    w = RNG.normal(1, 0.1, 257)
    assert np.allclose(oracle.rmsnorm(h, w, 0.0), y * w, rtol=1e-14, atol=1e-15)


# --------------------------------------------------------------------- rope
def test_rope_position_zero_and_unit_rotations():
    x = RNG.normal(0, 1, (3, 2, D))
    assert np.array_equal(oracle.rope(x, [0, 0, 0], 1e6), x)
    # pair 0 at position 1 turns by exactly 1 radian; pair 1 by theta^(-2/128)
    e = np.zeros((1, 1, D))
    e[0, 0, 0] = 1.0
    y = oracle.rope(e, [1], 1e6)[0, 0]
    assert y[0] == pytest.approx(math.cos(1.0), abs=1e-15) and y[64] == pytest.approx(math.sin(1.0), abs=1e-15)
    assert np.count_nonzero(y) == 2
    e = np.zeros((1, 1, D))
    e[0, 0, 65] = 1.0  # the second element of pair 1
    a1 = 10.0 ** (-6.0 / 64.0)  # (10^6)^(-2/128)
    y = oracle.rope(e, [1], 1e6)[0, 0]
    assert y[1] == pytest.approx(-math.sin(a1), abs=1e-15) and y[65] == pytest.approx(math.cos(a1), abs=1e-15)


def test_rope_is_complex_multiplication():
    x = RNG.normal(0, 1, (5, 3, D))
    pos = np.array([0, 1, 17, 4095, 32767])
    theta = 1e6
    y = oracle.rope(x, pos, theta)
    z = x[:, :, :64] + 1j * x[:, :, 64:]
    freq = theta ** (-np.arange(64) * 2.0 / D)
    zr = z * np.exp(1j * pos[:, None, None] * freq[None, None, :])
    # the two fp64 angles differ by a few ulps of pos * freq (pos up to 2^15)
    assert np.allclose(y[:, :, :64], zr.real, rtol=0, atol=1e-11)
    assert np.allclose(y[:, :, 64:], zr.imag, rtol=0, atol=1e-11)
    # each pair keeps its length
    assert np.allclose(np.abs(z), np.hypot(y[:, :, :64], y[:, :, 64:]), rtol=1e-13)


def test_rope_scores_depend_on_relative_position_only():
    q = RNG.normal(0, 1, (1, 1, D))
    k = RNG.normal(0, 1, (1, 1, D))
    for a, b, t in ((5, 2, 100), (0, 9, 7), (300, 301, 1000)):
        s1 = np.sum(oracle.rope(q, [a], 1e4) * oracle.rope(k, [b], 1e4))
        s2 = np.sum(oracle.rope(q, [a + t], 1e4) * oracle.rope(k, [b + t], 1e4))
        assert s1 == pytest.approx(s2, rel=1e-11, abs=1e-11)


# ---------------------------------------------------------------- attention
def test_attention_single_key_and_uniform_scores():
    kc = RNG.normal(0, 1, (2, 6, D))
    vc = RNG.normal(0, 1, (2, 6, D))
    q = RNG.normal(0, 1, (1, 4, D))
    out = oracle.attention(q, kc, vc, [0])
    for h in range(4):
        assert np.array_equal(out[0, h], vc[h // 2, 0])
    # q = 0: every allowed key has the same score -> mean of the values
    out = oracle.attention(np.zeros((2, 4, D)), kc, vc, [3, 5])
    for h in range(4):
        assert np.allclose(out[0, h], vc[h // 2, :4].mean(axis=0), rtol=1e-14, atol=1e-15)
        assert np.allclose(out[1, h], vc[h // 2, :6].mean(axis=0), rtol=1e-14, atol=1e-15)


def test_attention_two_keys_exact_weights():
    # scores 0 and ln 3 after the 1/sqrt(128) scale: weights exactly 1/4 and 3/4
    q = np.zeros((1, 1, D))
    q[0, 0, 3] = 2.0
    kc = np.zeros((1, 2, D))
    kc[0, 1, 3] = math.log(3.0) * math.sqrt(D) / 2.0
    vc = RNG.normal(0, 1, (1, 2, D))
    out = oracle.attention(q, kc, vc, [1])
    assert np.allclose(out[0, 0], 0.25 * vc[0, 0] + 0.75 * vc[0, 1], rtol=1e-13, atol=1e-15)


def test_attention_group_mapping_and_causality():
    hq, hkv, L = 6, 3, 9
    kc = RNG.normal(0, 1, (hkv, L, D))
    vc = np.zeros((hkv, L, D))
    for g in range(hkv):
        vc[g] = g + 1.0  # the value identifies the kv head
    q = RNG.normal(0, 1, (2, hq, D))
    out = oracle.attention(q, kc, vc, [4, 8])
    for h in range(hq):
        assert np.allclose(out[:, h], h // 2 + 1.0, rtol=1e-14)
    # entries after a row's position do not reach it
    vc2 = RNG.normal(0, 1, (hkv, L, D))
    a = oracle.attention(q, kc, vc2, [4, 8])
    kc_b, vc_b = kc.copy(), vc2.copy()
    kc_b[:, 5:] = RNG.normal(0, 5, (hkv, L - 5, D))
    vc_b[:, 5:] = RNG.normal(0, 5, (hkv, L - 5, D))
    b = oracle.attention(q, kc_b, vc_b, [4, 8])
    assert np.array_equal(a[0], b[0]) and not np.allclose(a[1], b[1])


# --------------------------------------------------------------------- silu
def test_silu_mul_against_scipy():
    g = RNG.normal(0, 4, (3, 50))
    u = RNG.normal(0, 1, (3, 50))
    out = oracle.silu_mul(np.concatenate([g, u], axis=1))
    assert np.allclose(out, g * special.expit(g) * u, rtol=1e-14, atol=1e-300)
    s = oracle.silu_mul(np.array([[0.0, 3.0, -3.0, -800.0] + [1.0] * 4]))[0]
    assert s[0] == 0.0 and s[3] == 0.0
    assert s[1] - s[2] == pytest.approx(3.0, rel=1e-15)  # silu(x) - silu(-x) = x


# --------------------------------------------------- model, cache and round
def small_params(dims: od.Dims, seed: int) -> dict:
    r = np.random.default_rng(seed)
    n_qkv = dims.q_dim + 2 * dims.kv_dim
    p = {"embed": r.normal(0, 1.0, (dims.vocab, dims.hidden)).astype(np.float16),
         "final_norm": r.normal(1, 0.1, dims.hidden).astype(np.float16),
         "lm_head": r.normal(0, 0.05, (dims.vocab, dims.hidden)).astype(np.float16)}
    for l in range(dims.layers):
        p[f"{l}.in_norm"] = r.normal(1, 0.1, dims.hidden).astype(np.float16)
        p[f"{l}.qkv"] = r.normal(0, 0.05, (n_qkv, dims.hidden)).astype(np.float16)
        p[f"{l}.qkv_bias"] = r.normal(0, 0.1, n_qkv).astype(np.float16)
        p[f"{l}.o"] = r.normal(0, 0.05, (dims.hidden, dims.q_dim)).astype(np.float16)
        p[f"{l}.post_norm"] = r.normal(1, 0.1, dims.hidden).astype(np.float16)
        p[f"{l}.gate_up"] = r.normal(0, 0.05, (2 * dims.inter, dims.hidden)).astype(np.float16)
        p[f"{l}.down"] = r.normal(0, 0.05, (dims.hidden, dims.inter)).astype(np.float16)
    return p


DIMS = od.Dims(layers=2, hidden=256, inter=384, q_heads=4, kv_heads=2, vocab=300, theta=1e4)


def test_incremental_decode_matches_one_pass_and_is_causal():
    params = small_params(DIMS, 1)
    model = od.Model(DIMS, params, "f16")
    toks = RNG.integers(0, DIMS.vocab, (2, 11))
    pos = np.broadcast_to(np.arange(11), (2, 11))
    full = od.forward(model, od.Cache(DIMS, 2, 16), toks, pos)
    cache = od.Cache(DIMS, 2, 16)
    for t in range(11):
        step = od.forward(model, cache, toks[:, t:t + 1], pos[:, t:t + 1])
        assert np.allclose(step[:, 0], full[:, t], rtol=0, atol=1e-9)
    # a later token does not reach earlier rows
    toks2 = toks.copy()
    toks2[:, 7] = (toks2[:, 7] + 1) % DIMS.vocab
    full2 = od.forward(model, od.Cache(DIMS, 2, 16), toks2, pos)
    assert np.allclose(full2[:, :7], full[:, :7], rtol=0, atol=1e-12)
    assert not np.allclose(full2[:, 7], full[:, 7])


def greedy_decode(model, prompt, steps, capacity):
    """Plain greedy decoding through the cache, one token at a time."""
    B, Lp = prompt.shape
    cache = od.Cache(model.dims, B, capacity)
    pos = np.broadcast_to(np.arange(Lp), (B, Lp))
    logits = od.forward(model, cache, prompt, pos)[:, -1]
    out = []
    for t in range(steps):
        tok = np.argmax(logits.astype(np.float32), axis=1)
        out.append(tok)
        logits = od.forward(model, cache, tok[:, None], np.full((B, 1), Lp + t))[:, 0]
    return np.stack(out, 1)


@pytest.mark.parametrize("variant", ["int4", "fp8"])
def test_greedy_speculation_emits_the_parent_greedy_decode(variant):
    params = small_params(DIMS, 2)
    parent = od.Model(DIMS, params, "f16")
    draft = od.Model(DIMS, params, variant)
    B, Lp, k, cap = 2, 6, 4, 64
    prompt = RNG.integers(0, DIMS.vocab, (B, Lp))
    dc, pc = od.Cache(DIMS, B, cap), od.Cache(DIMS, B, cap)
    st = od.prefill([draft, parent], [dc, pc], prompt)
    n_hist = []
    for _ in range(6):
        res = od.spec_round(draft, parent, dc, pc, st, k, None, None, temperature=0.0)
        n_hist.extend(res["n_accepted"].tolist())
    steps = min(len(e) for e in st.emitted)
    ref = greedy_decode(parent, prompt, steps, cap)
    for b in range(B):
        assert st.emitted[b][:steps] == ref[b].tolist()
    # rejections happened (the rollback was exercised) and some drafts were accepted
    assert min(n_hist) < k and max(n_hist) > 0
    # after the rounds, every cache position before the pending token holds what
    # one pass over the committed tokens writes there
    for b in range(B):
        seq = np.concatenate([prompt[b], np.array(st.emitted[b][:-1])])
        assert len(seq) == st.pos[b]
        c = od.Cache(DIMS, 1, cap)
        od.forward(parent, c, seq[None, :], np.arange(len(seq))[None, :])
        n = len(seq)
        assert np.allclose(pc.k[:, b, :, :n], c.k[:, 0, :, :n], rtol=0, atol=2e-3)
        assert np.allclose(pc.v[:, b, :, :n], c.v[:, 0, :, :n], rtol=0, atol=2e-3)
        c2 = od.Cache(DIMS, 1, cap)
        od.forward(draft, c2, seq[None, :n - 1], np.arange(n - 1)[None, :])
        assert np.allclose(dc.k[:, b, :, :n - 1], c2.k[:, 0, :, :n - 1], rtol=0, atol=2e-3)


def test_identical_draft_accepts_every_token():
    params = small_params(DIMS, 3)
    m = od.Model(DIMS, params, "f16")
    B, k = 2, 3
    prompt = RNG.integers(0, DIMS.vocab, (B, 4))
    dc, pc = od.Cache(DIMS, B, 32), od.Cache(DIMS, B, 32)
    st = od.prefill([m, m], [dc, pc], prompt)
    for r in range(3):
        ud = RNG.integers(0, 1 << 24, (k, B))
        ua = RNG.integers(0, 1 << 24, (B, k + 1))
        res = od.spec_round(m, m, dc, pc, st, k, ud, ua, temperature=1.0)
        assert np.all(res["n_accepted"] == k)
    assert st.pos.tolist() == [3 + 3 * (k + 1)] * B


@pytest.mark.parametrize("variant", ["int4", "fp8"])
def test_greedy_speculation_with_chains_emits_the_parent_greedy_decode(variant):
    params = small_params(DIMS, 4)
    parent = od.Model(DIMS, params, "f16")
    draft = od.Model(DIMS, params, variant)
    B, c, Lp, k, cap = 2, 3, 5, 3, 64
    prompt = RNG.integers(0, DIMS.vocab, (B, Lp))
    dc, pc = od.Cache(DIMS, B * c, cap), od.Cache(DIMS, B * c, cap)
    st = od.prefill_chains([draft, parent], [dc, pc], prompt, c)
    for _ in range(5):
        od.spec_round_multi(draft, parent, dc, pc, st, c, k, None, None, temperature=0.0)
    steps = min(len(e) for e in st.emitted)
    ref = greedy_decode(parent, prompt, steps, cap)
    for b in range(B):
        assert st.emitted[b][:steps] == ref[b].tolist()
        seq = np.concatenate([prompt[b], np.array(st.emitted[b][:-1])])
        n = len(seq)
        one = od.Cache(DIMS, 1, cap)
        od.forward(parent, one, seq[None, :], np.arange(n)[None, :])
        for j in range(c):  # every chain of the sequence holds the committed prefix
            assert np.allclose(pc.k[:, b * c + j, :, :n], one.k[:, 0, :, :n], rtol=0, atol=2e-3)


def test_chains_with_an_identical_draft_accept_every_token():
    """Several chains at T = 1: a draft identical to the parent accepts every
    token, from the lowest chain."""
    params = small_params(DIMS, 5)
    parent = od.Model(DIMS, params, "f16")
    B, c, k = 2, 3, 3
    prompt = RNG.integers(0, DIMS.vocab, (B, 4))
    dc, pc = od.Cache(DIMS, B * c, 32), od.Cache(DIMS, B * c, 32)
    st = od.prefill_chains([parent, parent], [dc, pc], prompt, c)
    for _ in range(2):
        ud = RNG.integers(0, 1 << 24, (k, B * c))
        ua = RNG.integers(0, 1 << 24, (B, c * k + 1))
        res = od.spec_round_multi(parent, parent, dc, pc, st, c, k, ud, ua, temperature=1.0)
        assert (res["n_accepted"] == k).all() and (res["chain"] == 0).all()
