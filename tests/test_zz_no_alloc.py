"""The allocation-free accept call (sq_spec_accept_noalloc) against
sq_spec_accept: two calls in a row, the second smaller, in every mode
(stochastic with the distributions returned, greedy, the plain sampler);
results bit for bit equal, and checked against the oracle on the kernel's own
distributions.  Then the call captured in a HIP graph: every replay, with
eager work and synchronisations in between, gives the eager results."""
import pytest
import torch

import paper_2609_21704_amd as sq
from accept_compare import check_accept
from paper_2609_21704_amd import synth

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _case(b, kd, v, seed):
    draft = synth.normal_f32((kd, b, v), 2.0, synth.stream_seed(seed, 1))
    target = torch.empty((b, kd + 1, v), dtype=torch.float32)
    target[:, :kd] = draft.permute(1, 0, 2) + synth.normal_f32((b, kd, v), 0.5, synth.stream_seed(seed, 2))
    target[:, kd] = synth.normal_f32((b, v), 2.0, synth.stream_seed(seed, 3))
    tok = synth.tokens((kd, b), v, synth.stream_seed(seed, 4))
    u24 = synth.uniform_u24((b, kd + 1), synth.stream_seed(seed, 5))
    return draft, target, tok, u24


def _both(b, kd, v, temp, seed):
    draft, target, tok, u24 = _case(b, kd, v, seed)
    d = draft.to(DEV) if kd > 0 else None
    tg, tk, uu = target.to(DEV), tok.to(DEV) if kd > 0 else None, u24.to(DEV)
    want = temp > 0
    outs = []
    for fn in (sq.sq_spec_accept, sq.sq_spec_accept_noalloc):
        q_out = torch.full((kd, b, v), -1.0, device=DEV) if want and kd > 0 else None
        p_out = torch.full((b, kd + 1, v), -1.0, device=DEV) if want else None
        n = torch.full((b,), -7, dtype=torch.int32, device=DEV)
        t = torch.full((b,), -7, dtype=torch.int32, device=DEV)
        fn(d, tg, tk, uu, temp, n_accepted=n, next_token=t, q_out=q_out, p_out=p_out)
        torch.cuda.synchronize()
        outs.append((n, t, q_out, p_out))
    (n0, t0, q0, p0), (n1, t1, q1, p1) = outs
    assert torch.equal(n0, n1) and torch.equal(t0, t1)
    if want:
        assert torch.equal(p0, p1) and (kd == 0 or torch.equal(q0, q1))
    check_accept(draft.numpy(), target.numpy(), tok.numpy(), u24.numpy(), temp, n1.cpu().numpy(), t1.cpu().numpy(),
                 q1.cpu().numpy() if want and kd > 0 else None, p1.cpu().numpy() if want else None)
    return n1, t1


@pytest.mark.parametrize("temp", [1.0, 0.0])
def test_noalloc_matches_spec_accept_two_calls_second_smaller(temp):
    # the second call needs less scratch than the first: what the first left in
    # the shared array must not leak into it
    _both(8, 8, 151936, temp, 11)
    _both(1, 4, 4096, temp, 12)


def test_noalloc_plain_sampler_and_largest_within_the_array():
    _both(3, 0, 151936, 1.0, 13)                 # kd = 0: a draft-token draw
    _both(96, 8, 151936, 1.0, 14)                # 4.1 MB of the 4 MiB array (97 sequences at most)
    _both(1, 1, 5, 1.0, 15)


def test_noalloc_inside_a_captured_graph():
    b, kd, v = 4, 8, 151936
    draft, target, tok, u24 = _case(b, kd, v, 16)
    d, tg, tk, uu = draft.to(DEV), target.to(DEV), tok.to(DEV), u24.to(DEV)
    n = torch.zeros((b,), dtype=torch.int32, device=DEV)
    t = torch.zeros((b,), dtype=torch.int32, device=DEV)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        sq.sq_spec_accept_noalloc(d, tg, tk, uu, 1.0, n_accepted=n, next_token=t)
    for r in range(4):
        uu.copy_(synth.uniform_u24((b, kd + 1), 100 + r, DEV))
        g.replay()
        torch.cuda.synchronize()
        got = (n.clone(), t.clone())
        n_ref, t_ref = sq.sq_spec_accept(d, tg, tk, uu, 1.0)   # eager, on the library workspace
        _both(2, 3, 5000, 1.0, 200 + r)                          # other eager work on the shared array
        torch.cuda.synchronize()
        assert torch.equal(got[0], n_ref) and torch.equal(got[1], t_ref), r
