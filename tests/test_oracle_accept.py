"""Pins of the oracle's softmax and speculative accept / resample step (token
acceptance or correction, SpecQuant SS III-D.4; guess-set rule of SS III-A)
against scipy, exact enumeration of the output distribution at V = 8,
chi-square tests over 10^6 sequences, the closed-form acceptance law
P(n >= i) = prod_{j<i} beta_j, and the greedy (T = 0) special case."""
import numpy as np
import pytest
from scipy import special, stats

import oracle

RNG = np.random.default_rng(2024)
U = 1 << 24


# --------------------------------------------------------------- softmax ---
def test_softmax_matches_scipy_and_identities():
    l = RNG.normal(0, 2, (5, 1000)).astype(np.float32)
    for T in (1.0, 0.7, 2.5):
        p = oracle.softmax(l, T)
        ref = special.softmax(l.astype(np.float64) / T, axis=1)
        assert np.max(np.abs(p - ref)) < 1e-15
        assert np.allclose(p.sum(axis=1), 1.0, rtol=0, atol=1e-12)
    # uniform logits -> 1/V
    assert np.allclose(oracle.softmax(np.full((1, 4096), 3.25, np.float32)), 1 / 4096, rtol=1e-14, atol=0)
    # shift invariance (logits on a 2^-8 grid, so adding 64 is exact in fp32)
    lg = (np.round(l * 256) / 256).astype(np.float32)
    assert np.array_equal(lg + np.float32(64.0) - np.float32(64.0), lg)
    assert np.allclose(oracle.softmax(lg + np.float32(64.0)), oracle.softmax(lg), rtol=1e-12, atol=1e-300)
    # one huge logit -> one-hot
    h = np.zeros((1, 50), np.float32)
    h[0, 17] = 1e4
    p = oracle.softmax(h)
    assert p[0, 17] == 1.0 and np.count_nonzero(p) == 1


# ---------------------------------------------------------- helpers -------
def _accept_one(dl, tl, x, u0, u1, T=1.0):
    """kd = 1, b = 1: draft logits [v], target logits [2][v]."""
    n, t, _, _ = oracle.spec_accept(dl[None, None, :], tl[None, :, :], np.array([[x]], np.int32),
                                    np.array([[u0, u1]], np.uint32), T)
    return int(n[0]), int(t[0])


def _threshold(pred):
    """Smallest u24 in [0, 2^24] for which pred(u24) is False; pred monotone."""
    lo, hi = 0, U
    while lo < hi:
        mid = (lo + hi) // 2
        if pred(mid):
            lo = mid + 1
        else:
            hi = mid
    return lo


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_exact_enumeration_emitted_token_law_equals_target(seed):
    """P(emit y) = sum_x q(x) [min(1,p/q)(x) 1{y=x} + (1 - min(1,p/q)(x)) res(y)] = p(y)."""
    rng = np.random.default_rng(seed)
    v = 8
    dl = rng.normal(0, 1.5, v).astype(np.float32)
    tl = np.stack([dl + rng.normal(0, 1.0, v), rng.normal(0, 1, v)]).astype(np.float32)
    q = special.softmax(dl.astype(np.float64))
    p = special.softmax(tl[0].astype(np.float64))
    # acceptance count A(x): u24 values for which x is accepted (accept iff u24 < A)
    A = np.array([_threshold(lambda u, x=x: _accept_one(dl, tl, x, u, 0)[0] == 1) for x in range(v)], np.float64)
    assert np.all(np.abs(A / U - np.minimum(1.0, p / q)) <= 2.0 / U)
    # residual law: reject a token with p < q, then read off token(u_final) boundaries
    xr = int(np.argmax(q - p))
    assert _accept_one(dl, tl, xr, U - 1, 0)[0] == 0
    bounds = [0] + [_threshold(lambda u, y=y: _accept_one(dl, tl, xr, U - 1, u)[1] < y) for y in range(1, v)] + [U]
    res = np.diff(np.array(bounds, np.float64)) / U
    r = np.maximum(p - q, 0)
    assert np.all(np.abs(res - r / r.sum()) <= 2.0 / U)
    emit = q * (A / U) + (q * (1 - A / U)).sum() * res
    assert np.max(np.abs(emit - p)) < 1e-6


def test_bonus_token_law_when_all_accepted():
    v = 8
    rng = np.random.default_rng(7)
    dl = rng.normal(0, 1, v).astype(np.float32)
    tl = np.stack([dl, rng.normal(0, 1, v)]).astype(np.float32)   # p_0 = q_0: always accepted
    p1 = special.softmax(tl[1].astype(np.float64))
    for x in range(v):
        assert _accept_one(dl, tl, x, U - 1, 0)[0] == 1
    bounds = [0] + [_threshold(lambda u, y=y: _accept_one(dl, tl, 3, 0, u)[1] < y) for y in range(1, v)] + [U]
    res = np.diff(np.array(bounds, np.float64)) / U
    assert np.max(np.abs(res - p1)) <= 2.0 / U


def _sample(probs, u):
    """Inverse-CDF draw per row of probs with uniforms u (test-side sampler)."""
    c = np.cumsum(probs, axis=-1)
    return np.minimum((u[..., None] >= c).sum(axis=-1), probs.shape[-1] - 1)


def test_chi_square_kd4_positions_and_acceptance_law():
    """b = 10^6 sequences, kd = 4 distinct rows at V = 8."""
    rng = np.random.default_rng(11)
    b, kd, v = 1_000_000, 4, 8
    dl = rng.normal(0, 1.2, (kd, v)).astype(np.float32)
    tl = np.concatenate([dl + rng.normal(0, 0.8, (kd, v)).astype(np.float32),
                         rng.normal(0, 1, (1, v)).astype(np.float32)])
    q = special.softmax(dl.astype(np.float64), axis=1)
    p = special.softmax(tl.astype(np.float64), axis=1)
    x = _sample(q[None, :, :], rng.random((b, kd))).astype(np.int32)          # [b][kd]
    u24 = rng.integers(0, U, (b, kd + 1), dtype=np.uint32)
    draft = np.broadcast_to(dl[:, None, :], (kd, b, v))
    target = np.broadcast_to(tl[None, :, :], (b, kd + 1, v))
    n, nxt, _, _ = oracle.spec_accept(draft, target, np.ascontiguousarray(x.T), u24, 1.0)
    crit = lambda dof: stats.chi2.ppf(1 - 1e-3, dof)
    # acceptance law: P(n = i) = prod_{j<i} beta_j (1 - beta_i), P(n = kd) = prod beta
    beta = np.minimum(p[:kd], q).sum(axis=1)
    law = np.array([np.prod(beta[:i]) * (1 - beta[i]) for i in range(kd)] + [np.prod(beta)])
    obs = np.bincount(n, minlength=kd + 1)
    assert np.sum((obs - b * law) ** 2 / (b * law)) < crit(kd)
    # emitted token at each position, given the position is reached, follows p_i
    for i in range(kd + 1):
        reached = n >= i
        tok = np.where(n[reached] > i, x[reached, min(i, kd - 1)], nxt[reached])
        cnt = np.bincount(tok, minlength=v)
        exp = reached.sum() * p[i]
        assert np.sum((cnt - exp) ** 2 / exp) < crit(v - 1), i


def test_equal_distributions_accept_everything():
    b, kd, v = 64, 5, 300
    l = RNG.normal(0, 2, (kd + 1, v)).astype(np.float32)
    draft = np.broadcast_to(l[:kd, None, :], (kd, b, v))
    target = np.broadcast_to(l[None], (b, kd + 1, v))
    x = RNG.integers(0, v, (kd, b)).astype(np.int32)
    u24 = np.full((b, kd + 1), U - 1, np.uint32)
    n, nxt, _, _ = oracle.spec_accept(draft, target, x, u24, 1.0)
    assert np.all(n == kd)
    # bonus drawn from p_kd with u = 1 - 2^-24: the last token with mass
    assert np.all(nxt == np.nonzero(special.softmax(l[kd].astype(np.float64)) > 0)[0].max())


def test_zero_target_mass_always_rejects_and_out_of_range_token_rejects():
    v = 16
    dl = np.zeros(v, np.float32)
    tl = np.zeros((2, v), np.float32)
    tl[0, 3] = -1e30          # p_0(3) = 0 < q_0(3)
    for u in (0, 1, U // 2):
        n, tok = _accept_one(dl, tl, 3, u, u)
        assert n == 0 and tok != 3
    for bad in (-1, v, 1 << 30):
        n, _ = _accept_one(dl, tl, bad, 0, 0)
        assert n == 0


def test_greedy_rule_matches_argmax():
    """T = 0: accept iff x_i == argmax p_i; emit argmax at the first mismatch."""
    b, kd, v = 200, 4, 50
    tl = RNG.normal(0, 1, (b, kd + 1, v)).astype(np.float32)
    tl[0, 2, :] = 1.0                                    # all ties -> index 0
    am = tl.argmax(axis=2)
    x = am[:, :kd].copy().astype(np.int32)
    cut = RNG.integers(0, kd + 1, b)
    for s in range(b):
        if cut[s] < kd:
            x[s, cut[s]] = (am[s, cut[s]] + 1) % v
    draft = RNG.normal(0, 1, (kd, b, v)).astype(np.float32)
    n, nxt, _, _ = oracle.spec_accept(draft, tl, np.ascontiguousarray(x.T), None, 0.0)
    exp_n = np.array([next((i for i in range(kd) if x[s, i] != am[s, i]), kd) for s in range(b)])
    assert np.array_equal(n, exp_n)
    assert np.array_equal(nxt, am[np.arange(b), exp_n])
    assert am[0, 2] == 0


def test_one_hot_stochastic_reduces_to_greedy():
    """With one-hot p and q the stochastic rule is the paper's greedy rule."""
    b, kd, v = 100, 3, 20
    big = np.float32(1e4)
    pt = RNG.integers(0, v, (b, kd + 1))
    qt = np.where(RNG.random((b, kd)) < 0.5, pt[:, :kd], RNG.integers(0, v, (b, kd)))
    tl = np.zeros((b, kd + 1, v), np.float32)
    dl = np.zeros((kd, b, v), np.float32)
    for s in range(b):
        for i in range(kd + 1):
            tl[s, i, pt[s, i]] = big
        for i in range(kd):
            dl[i, s, qt[s, i]] = big
    x = np.ascontiguousarray(qt.T).astype(np.int32)
    u24 = RNG.integers(0, U, (b, kd + 1), dtype=np.uint32)
    n1, t1, _, _ = oracle.spec_accept(dl, tl, x, u24, 1.0)
    n0, t0, _, _ = oracle.spec_accept(dl, tl, x, None, 0.0)
    assert np.array_equal(n1, n0) and np.array_equal(t1, t0)


def test_kd0_is_a_plain_sampler():
    v = 8
    rng = np.random.default_rng(5)
    tl = rng.normal(0, 1, (1, 1, v)).astype(np.float32)
    p = special.softmax(tl[0, 0].astype(np.float64))
    bounds = [0]
    for y in range(1, v):
        bounds.append(_threshold(lambda u, y=y: oracle.spec_accept(None, tl, None, np.array([[u]], np.uint32))[1][0] < y))
    bounds.append(U)
    assert np.max(np.abs(np.diff(np.array(bounds, np.float64)) / U - p)) <= 2.0 / U


def test_pq_outputs_and_errors():
    b, kd, v = 3, 2, 40
    dl = RNG.normal(0, 1, (kd, b, v)).astype(np.float32)
    tl = RNG.normal(0, 1, (b, kd + 1, v)).astype(np.float32)
    x = RNG.integers(0, v, (kd, b)).astype(np.int32)
    u24 = RNG.integers(0, U, (b, kd + 1), dtype=np.uint32)
    n, t, q, p = oracle.spec_accept(dl, tl, x, u24, 0.9, want_pq=True)
    assert np.max(np.abs(q - special.softmax(dl.astype(np.float64) / 0.9, axis=2))) < 1e-15
    assert np.max(np.abs(p - special.softmax(tl.astype(np.float64) / 0.9, axis=2))) < 1e-15
    with pytest.raises(oracle.OracleError):
        oracle.spec_accept(dl, tl, x, u24, -1.0)
    with pytest.raises(oracle.OracleError):
        oracle.spec_accept(dl, tl, x, u24, 0.0, want_pq=True)
