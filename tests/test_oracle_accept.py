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


# ------------------------------------------- fp32 decisions, fallbacks, masks ---
from fractions import Fraction  # noqa: E402


def _law_of_final_draw(run):
    """Exact law of the token returned by run(u_final) over all 2^24 uniforms
    (the draw is monotone in u): P(token = y) for y = 0..v-1."""
    toks = {}
    lo = 0
    while lo < U:
        t = run(lo)
        hi = _threshold(lambda u, t=t: u < lo or run(u) <= t)  # first u with a larger token
        toks[t] = toks.get(t, 0) + (hi - lo)
        lo = hi
    return toks


def test_decisions_use_the_fp32_distributions_exactly():
    """The accept threshold over u24 is exactly ceil(2^24 p32(x) / q32(x)) for
    the fp32 roundings of p and q: checked with exact rational arithmetic."""
    rng = np.random.default_rng(17)
    v = 64
    for trial in range(6):
        dl = rng.normal(0, 1.5, v).astype(np.float32)
        tl = np.stack([dl + rng.normal(0, 0.7, v), rng.normal(0, 1, v)]).astype(np.float32)
        p32 = oracle.softmax(tl[0]).astype(np.float32)[0]
        q32 = oracle.softmax(dl).astype(np.float32)[0]
        x = int(np.argmax(q32 - p32)) if trial % 2 == 0 else int(rng.integers(0, v))
        ratio = Fraction(float(p32[x])) / Fraction(float(q32[x]))
        expect = U if ratio >= 1 else -(-ratio.numerator * U // ratio.denominator)   # ceil
        got = _threshold(lambda u: _accept_one(dl, tl, x, u, 0)[0] == 1)
        assert got == min(expect, U), (trial, got, expect)


def test_accept_probs_reproduces_spec_accept_from_its_fp32_distributions():
    rng = np.random.default_rng(23)
    b, kd, v = 40, 5, 700
    dl = rng.normal(0, 2, (kd, b, v)).astype(np.float32)
    tl = np.concatenate([dl.transpose(1, 0, 2) + rng.normal(0, 0.5, (b, kd, v)).astype(np.float32),
                         rng.normal(0, 2, (b, 1, v)).astype(np.float32)], axis=1)
    x = rng.integers(0, v, (kd, b)).astype(np.int32)
    u24 = rng.integers(0, U, (b, kd + 1), dtype=np.uint32)
    n, t, q, p = oracle.spec_accept(dl, tl, x, u24, 1.0, want_pq=True)
    n2, t2 = oracle.accept_probs(p.astype(np.float32), q.astype(np.float32), x, u24)
    assert np.array_equal(n, n2) and np.array_equal(t, t2)
    assert len(set(n.tolist())) > 2   # the case exercises several rejection positions


def _fallback_rows(v, rng):
    """A drafted row q0 whose residual max(0, p0 - q0) is positive at one token
    but below half a step of the 2^-60 grid, and p1 one-hot elsewhere."""
    p0 = rng.dirichlet(np.ones(v)).astype(np.float32)
    p0[0] += p0[1] + p0[2]                           # keep the row a distribution
    p0[1] = np.float32(2.0 ** -70)
    p0[2] = np.float32(2.0 ** -70 + 2.0 ** -93)      # exact in fp32: 2^-70 (1 + 2^-23)
    q0 = p0.copy()
    q0[1], q0[2] = p0[2], p0[1]                      # p0 - q0: -2^-93 at 1, +2^-93 at 2
    p1 = np.zeros(v, np.float32)
    p1[v - 1] = 1.0
    return p0, q0, p1


def test_zero_residual_on_the_grid_falls_back_to_p_n():
    """Rejecting token 1 (u q0(1) >= p0(1) for u = 1 - 2^-24) leaves a residual
    of 2^-93 at token 2, which is 0 on the 2^-60 grid: the draw falls back to
    p0 itself.  Its exact law over all 2^24 final uniforms is p0 (not p1, not
    the invalid token -1)."""
    rng = np.random.default_rng(29)
    v = 8
    p0, q0, p1 = _fallback_rows(v, rng)
    assert p0[2] - p0[1] == np.float32(2.0 ** -93) and q0[2] < p0[2]
    p = np.stack([p0, p1])[None]                     # [b=1][kd+1=2][v]
    q = q0[None, None]                               # [kd=1][b=1][v]

    def run(uf):
        n, t = oracle.accept_probs(p, q, np.array([[1]], np.int32), np.array([[U - 1, uf]], np.uint32))
        assert n[0] == 0
        return int(t[0])

    law = _law_of_final_draw(run)
    got = np.array([law.get(y, 0) for y in range(v)], np.float64) / U
    assert set(law) <= set(range(v))
    assert np.max(np.abs(got - p0.astype(np.float64))) <= 2.0 / U


def test_rejected_invalid_token_with_equal_rows_falls_back_to_p_n():
    """From logits: target row 0 equals draft row 0 and the drafted token is
    outside [0, v), so position 0 is rejected with an all-zero residual; the
    emitted token follows softmax(row 0), not row 1."""
    rng = np.random.default_rng(31)
    v = 8
    row0 = rng.normal(0, 1, v).astype(np.float32)
    row1 = np.full(v, -50.0, np.float32)
    row1[v - 1] = 50.0
    dl = row0[None, None]
    tl = np.stack([row0, row1])[None]
    p0 = special.softmax(row0.astype(np.float64))
    for bad in (-1, v):
        def run(uf, bad=bad):
            n, t, _, _ = oracle.spec_accept(dl, tl, np.array([[bad]], np.int32), np.array([[0, uf]], np.uint32))
            assert n[0] == 0
            return int(t[0])

        law = _law_of_final_draw(run)
        got = np.array([law.get(y, 0) for y in range(v)], np.float64) / U
        assert np.max(np.abs(got - p0)) <= 2.0 / U


def test_masked_logits_have_zero_probability():
    """-inf logits (masked tokens, here a whole block of 5000 of them) get
    probability 0: the rest is scipy's softmax over the finite logits; a
    drafted token masked in the parent is always rejected, and no masked token
    is ever emitted."""
    rng = np.random.default_rng(37)
    v = 9000
    tl = rng.normal(0, 2, (2, v)).astype(np.float32)
    dl = rng.normal(0, 2, v).astype(np.float32)
    tl[0, 1000:6000] = -np.inf
    tl[1, :4096] = -np.inf
    dl[7000:] = -np.inf
    p = oracle.softmax(tl)
    fin = np.isfinite(tl[0])
    assert np.all(p[0, ~fin] == 0)
    assert np.max(np.abs(p[0, fin] - special.softmax(tl[0, fin].astype(np.float64)))) < 1e-15
    assert np.all(oracle.softmax(dl)[0, 7000:] == 0)
    for u in (0, 12345, U - 1):
        for uf in (0, U // 3, U - 1):
            n, t = _accept_one(dl, tl, 2000, u, uf)     # p_0(2000) = 0 < q_0(2000)
            assert n == 0 and np.isfinite(tl[0, t])
            n, t = _accept_one(dl, tl, 500, 0, uf)       # u = 0: accepted, bonus row 1
            assert n == 1 and t >= 4096


@pytest.mark.parametrize("bad", ["nan", "+inf", "all-masked"])
def test_rows_without_a_distribution_invalidate_their_sequence(bad):
    rng = np.random.default_rng(41)
    b, kd, v = 4, 2, 100
    dl = rng.normal(0, 1, (kd, b, v)).astype(np.float32)
    tl = rng.normal(0, 1, (b, kd + 1, v)).astype(np.float32)
    x = rng.integers(0, v, (kd, b)).astype(np.int32)
    u24 = rng.integers(0, U, (b, kd + 1), dtype=np.uint32)
    val = {"nan": np.nan, "+inf": np.inf}.get(bad)
    if val is None:
        tl[1, 2, :] = -np.inf          # sequence 1: target row 2 fully masked
        dl[1, 2, :] = -np.inf          # sequence 2: draft row 1 fully masked
    else:
        tl[1, 2, 7] = val
        dl[1, 2, 9] = val
    n_ok, t_ok, _, _ = oracle.spec_accept(dl[:, [0, 3]], tl[[0, 3]], x[:, [0, 3]], u24[[0, 3]], 1.0)
    n, t, q, p = oracle.spec_accept(dl, tl, x, u24, 1.0, want_pq=True)
    assert n[1] == -1 and t[1] == -1 and n[2] == -1 and t[2] == -1
    assert np.array_equal(n[[0, 3]], n_ok) and np.array_equal(t[[0, 3]], t_ok)
    assert np.all(np.isnan(p[1, 2])) and np.all(np.isnan(q[1, 2])) and not np.any(np.isnan(p[0]))
    n2, t2 = oracle.accept_probs(p.astype(np.float32), q.astype(np.float32), x, u24)
    assert np.array_equal(n2, n) and np.array_equal(t2, t)
    # greedy reads the target rows only: sequence 1 is invalid, sequence 2 is not
    ng, tg, _, _ = oracle.spec_accept(dl, tl, x, None, 0.0)
    assert ng[1] == -1 and tg[1] == -1 and ng[2] >= 0 and tg[2] == int(np.argmax(tl[2, ng[2]]))
