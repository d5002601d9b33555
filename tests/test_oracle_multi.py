"""Pins of the multi-candidate acceptance oracle (several draft chains per
sequence, SS III-D.2; acceptance or correction, SS III-D.4): with one chain
it is the single-candidate rule bit for bit; with several chains the emitted
tokens follow the parent's distribution exactly (chi-square over 10^6 draws,
one token and two tokens deep through a prefix-dependent model); identical
draft and parent accept every token; the greedy form follows the argmax."""
import numpy as np
import pytest
from scipy import stats

import oracle

RNG = np.random.default_rng(11)
U = 1 << 24


def dirichlet(shape, v, alpha=0.7):
    return RNG.dirichlet(np.full(v, alpha), shape).astype(np.float32)


def test_one_chain_is_the_single_candidate_rule():
    for b, kd, v in ((64, 4, 300), (32, 1, 8), (16, 6, 5000)):
        p = dirichlet((b, kd + 1), v)
        q = dirichlet((kd, b), v)
        drafts = RNG.integers(0, v, (kd, b)).astype(np.int32)
        # some drafts drawn from q, some rows with p == q (full acceptance and the
        # zero-residual fallback), some out-of-range tokens
        for i in range(kd):
            for s in range(0, b, 3):
                drafts[i, s] = sample_chains(q[i, s], 1, 1)[0, 0]
        p[::5, 0] = q[0, ::5]
        drafts[0, 1] = -1
        drafts[kd - 1, 2] = v
        u = RNG.integers(0, U, (b, kd + 1)).astype(np.uint32)
        n1, t1 = oracle.accept_probs(p, q, drafts, u)
        n2, t2, ch = oracle.multi_accept_probs(p[:, None], q[:, :, None], drafts[:, :, None], u)
        assert np.array_equal(n1, n2) and np.array_equal(t1, t2)
        assert (ch == 0).all()
        assert len(set(n1.tolist())) > 1


def first_tokens(p, q, drafts, n, t, ch):
    """The first emitted token of each sequence."""
    b = len(n)
    return np.where(n >= 1, drafts[0, np.arange(b), ch], t)


def sample_chains(qrow, b, c):
    """[b][c] independent draws from the distribution qrow."""
    cdf = np.cumsum(qrow.astype(np.float64))
    return np.minimum(np.searchsorted(cdf / cdf[-1], RNG.random((b, c)), side="right"), len(qrow) - 1)


@pytest.mark.parametrize("c", [2, 3, 5])
def test_first_token_follows_the_parent(c):
    v, kd, b, reps = 6, 1, 200_000, 5
    p0 = np.array([0.30, 0.05, 0.25, 0.15, 0.15, 0.10], np.float32)
    q0 = np.array([0.10, 0.30, 0.10, 0.20, 0.05, 0.25], np.float32)
    counts = np.zeros(v)
    for _ in range(reps):
        x = sample_chains(q0, b, c).astype(np.int32)
        p = np.broadcast_to(p0, (b, c, kd + 1, v)).copy()
        q = np.broadcast_to(q0, (kd, b, c, v)).copy()
        drafts = x[None]
        u = RNG.integers(0, U, (b, c * kd + 1)).astype(np.uint32)
        n, t, ch = oracle.multi_accept_probs(p, q, drafts, u)
        y = first_tokens(p, q, drafts, n, t, ch)
        counts += np.bincount(y, minlength=v)
    p64 = p0.astype(np.float64)
    exp = p64 / p64.sum() * counts.sum()
    assert stats.chisquare(counts, exp).pvalue > 1e-4
    assert counts.sum() == b * reps


def test_two_tokens_follow_the_parent_through_the_tree():
    v, c, kd, b, reps = 4, 3, 2, 250_000, 4
    p0 = np.array([0.4, 0.1, 0.3, 0.2], np.float32)
    q0 = np.array([0.1, 0.4, 0.2, 0.3], np.float32)
    p1 = dirichlet((v,), v, 1.5)    # p(. | first token)
    q1 = dirichlet((v,), v, 1.5)
    counts = np.zeros((v, v))
    for _ in range(reps):
        x1 = sample_chains(q0, b, c)
        x2 = np.zeros_like(x1)
        for y in range(v):
            sel = x1 == y
            x2[sel] = sample_chains(q1[y], int(sel.sum()), 1)[:, 0]
        p = np.empty((b, c, kd + 1, v), np.float32)
        p[:, :, 0] = p0
        p[:, :, 1] = p1[x1]
        p[:, :, 2] = 1.0 / v
        q = np.empty((kd, b, c, v), np.float32)
        q[0] = q0
        q[1] = q1[x1]
        drafts = np.stack([x1, x2]).astype(np.int32)
        u = RNG.integers(0, U, (b, c * kd + 1)).astype(np.uint32)
        n, t, ch = oracle.multi_accept_probs(p, q, drafts, u)
        idx = np.arange(b)
        y1 = np.where(n >= 1, drafts[0, idx, ch], t)
        y2 = np.where(n >= 2, drafts[1, idx, ch], np.where(n == 1, t, -1))
        # sequences that emitted one token: a second round at the node y1
        redo = np.nonzero(y2 < 0)[0]
        m = len(redo)
        x1b = np.zeros((m, c), np.int64)
        for y in range(v):
            sel = y1[redo] == y
            x1b[sel] = sample_chains(q1[y], int(sel.sum()), c)
        pb = np.empty((m, c, 2, v), np.float32)
        pb[:, :, 0] = p1[y1[redo]][:, None, :]
        pb[:, :, 1] = 1.0 / v
        qb = np.broadcast_to(q1[y1[redo]][None, :, None, :], (1, m, c, v)).copy()
        ub = RNG.integers(0, U, (m, c + 1)).astype(np.uint32)
        nb, tb, chb = oracle.multi_accept_probs(pb, qb, x1b[None].astype(np.int32), ub)
        y2[redo] = np.where(nb >= 1, x1b[np.arange(m), chb], tb)
        np.add.at(counts, (y1, y2), 1)
    a0, a1 = p0.astype(np.float64), p1.astype(np.float64)
    exp = (a0[:, None] / a0.sum()) * (a1 / a1.sum(1, keepdims=True))
    exp = exp / exp.sum() * counts.sum()
    assert stats.chisquare(counts.ravel(), exp.ravel()).pvalue > 1e-4


def test_identical_draft_accepts_everything_and_nan_rows_are_invalid():
    b, c, kd, v = 20, 4, 5, 100
    rows = dirichlet((b, c, kd + 1), v)
    q = np.ascontiguousarray(np.transpose(rows[:, :, :kd], (2, 0, 1, 3)))
    drafts = RNG.integers(0, v, (kd, b, c)).astype(np.int32)
    for d in range(kd):
        for s in range(b):
            for j in range(c):
                drafts[d, s, j] = sample_chains(q[d, s, j], 1, 1)[0, 0]
    u = RNG.integers(0, U, (b, c * kd + 1)).astype(np.uint32)
    n, t, ch = oracle.multi_accept_probs(rows, q, drafts, u)
    assert (n == kd).all() and (ch == 0).all()
    rows[3, 2, 1, 7] = np.nan
    n, t, ch = oracle.multi_accept_probs(rows, q, drafts, u)
    assert n[3] == -1 and t[3] == -1 and ch[3] == -1 and (n[:3] == kd).all()


def test_greedy_follows_the_argmax():
    b, c, kd, v = 3, 3, 2, 10
    logits = RNG.normal(0, 1, (b, c, kd + 1, v)).astype(np.float32)
    drafts = np.zeros((kd, b, c), np.int32)
    g0 = np.argmax(logits[:, 0, 0], axis=1)
    # sequence 0: chain 2 has the argmax at depth 0, then matches at depth 1 too
    drafts[0, 0] = [(g0[0] + 1) % v, (g0[0] + 2) % v, g0[0]]
    logits[0, 2, 1] = logits[0, 0, 1]  # its depth-1 row
    drafts[1, 0, 2] = np.argmax(logits[0, 2, 1])
    # sequence 1: no chain has the argmax
    drafts[0, 1] = (g0[1] + 1) % v
    # sequence 2: chains 0 and 1 agree at depth 0, only chain 1 at depth 1
    drafts[0, 2] = [g0[2], g0[2], (g0[2] + 3) % v]
    logits[2, 1] = logits[2, 0]
    drafts[1, 2] = [(np.argmax(logits[2, 0, 1]) + 1) % v, np.argmax(logits[2, 0, 1]), 0]
    n, t, ch = oracle.multi_accept_greedy(logits, drafts)
    assert n.tolist() == [2, 0, 2]
    assert ch.tolist() == [2, 0, 1]
    assert t[0] == np.argmax(logits[0, 2, 2]) and t[1] == g0[1] and t[2] == np.argmax(logits[2, 1, 2])
    # one chain: the single-candidate greedy rule
    n1, t1, _, _ = oracle.spec_accept(None if kd == 0 else np.zeros((kd, b, v), np.float32), logits[:, 0],
                                      drafts[:, :, 0], None, 0.0)
    n2, t2, _ = oracle.multi_accept_greedy(logits[:, :1], drafts[:, :, :1])
    assert np.array_equal(n1, n2) and np.array_equal(t1, t2)
