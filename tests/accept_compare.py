"""Comparison of the GPU accept step with the oracle (test helper).

The kernel takes its decisions and draws on fp32 distributions; so does the
oracle, on the fp32 roundings of its own fp64 softmax.  Two checks follow:
  1. exact: the oracle's rule applied to the kernel's own fp32 distributions
     (q_out / p_out) gives the kernel's n_accepted and next_token bit for bit;
  2. end to end: every fp32 probability of the kernel equals the oracle's
     fp32 rounding of its fp64 value or is one ulp away (the two fp64 values
     differ in the last bits: another exp and another summation order).  A
     sequence whose fp32 rows all agree bit for bit must then get the
     oracle's end-to-end decisions and draw exactly; only a sequence with a
     differing element may differ, and such sequences are counted.
"""
import numpy as np

import oracle


def ulps(a32, b32):
    """Distance in units in the last place between non-negative fp32 arrays
    (NaN against NaN counts 0, NaN against a number a huge distance)."""
    a = np.asarray(a32, np.float32)
    b = np.asarray(b32, np.float32)
    d = np.abs(a.view(np.int32).astype(np.int64) - b.view(np.int32).astype(np.int64))
    na, nb = np.isnan(a), np.isnan(b)
    d[na & nb] = 0
    d[na ^ nb] = 1 << 40
    return d


def check_accept(draft, target, tok, u24, temp, n_gpu, t_gpu, q_out=None, p_out=None):
    """Both checks; draft [kd][b][v], target [b][kd+1][v], tok [kd][b], u24
    [b][kd+1] and the kernel's q_out [kd][b][v] / p_out [b][kd+1][v] as numpy
    arrays (the distributions are required at T > 0).  Returns the number of
    sequences whose fp32 rows differ from the oracle's somewhere."""
    b, kd1, v = target.shape
    kd = kd1 - 1
    if temp == 0.0:
        n_ref, t_ref, _, _ = oracle.spec_accept(draft, target, tok, None, 0.0)
        assert np.array_equal(n_gpu, n_ref) and np.array_equal(t_gpu, t_ref)
        return 0
    assert p_out is not None and (kd == 0 or q_out is not None), "the kernel's distributions are needed"
    u32 = np.asarray(u24).view(np.uint32)
    n1, t1 = oracle.accept_probs(p_out, q_out, tok, u32)
    assert np.array_equal(n_gpu, n1), "decisions differ from the rule on the kernel's own fp32 distributions"
    assert np.array_equal(t_gpu, t1), "draws differ from the rule on the kernel's own fp32 distributions"
    n_ref, t_ref, q_ref, p_ref = oracle.spec_accept(draft, target, tok, u32, temp, want_pq=True)
    dp = ulps(p_out, p_ref.astype(np.float32))
    assert dp.max() <= 1, dp.max()
    differs = (dp > 0).any(axis=(1, 2))
    count, total = int((dp > 0).sum()), dp.size
    if kd > 0:
        dq = ulps(q_out, q_ref.astype(np.float32))
        assert dq.max() <= 1, dq.max()
        differs |= (dq > 0).any(axis=(0, 2))
        count, total = count + int((dq > 0).sum()), total + dq.size
    assert count <= max(8, total // 100000), (count, total)   # a last-bit flip is rare
    mismatch = (n_gpu != n_ref) | (t_gpu != t_ref)
    assert not np.any(mismatch & ~differs), np.nonzero(mismatch & ~differs)[0][:10]
    return int(differs.sum())
