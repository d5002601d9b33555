"""GPU parity of multi-candidate drafting (several draft chains per sequence,
SS III-D.2; acceptance or correction over them, SS III-D.4): the accept
kernel against the oracle's rule on the kernel's own fp32 distributions (bit
for bit) and end to end from the logits; one chain equal to the
single-candidate call; greedy; rows without a distribution; the cache
adoption and the commit."""
import numpy as np
import pytest
import torch

import oracle

import paper_2609_21704_amd as sq

pytestmark = pytest.mark.gpu
DEV = "cuda"
U = 1 << 24


def gen(seed):
    g = torch.Generator(device="cpu")
    g.manual_seed(seed)
    return g


def make_case(b, c, kd, v, seed, share=0.5, noise=0.3):
    """Draft logits N(0, 2); target = draft + N(0, noise); chain tokens drawn
    from the draft rows, a chain repeating the previous chain's token with
    probability `share` (so that several chains stay alive together)."""
    g = gen(seed)
    rng = np.random.default_rng(seed)
    dl = (torch.randn((kd, b, c, v), generator=g) * 2).float()
    tl = torch.empty((b, c, kd + 1, v))
    tl[:, :, :kd] = dl.permute(1, 2, 0, 3) + noise * torch.randn((b, c, kd, v), generator=g)
    tl[:, :, kd] = torch.randn((b, c, v), generator=g) * 2
    q = oracle.softmax(dl.reshape(-1, v).numpy()).reshape(kd, b, c, v) if kd else None
    tok = np.zeros((kd, b, c), np.int32)
    for d in range(kd):
        for s in range(b):
            for j in range(c):
                if j > 0 and rng.random() < share:
                    tok[d, s, j] = tok[d, s, j - 1]
                else:
                    cdf = np.cumsum(q[d, s, j])
                    tok[d, s, j] = min(int(np.searchsorted(cdf / cdf[-1], rng.random(), side="right")), v - 1)
    u = torch.randint(0, U, (b, c * kd + 1), generator=g, dtype=torch.int64).to(torch.int32)
    return dl, tl.contiguous(), torch.from_numpy(tok), u


CASES = [(1, 4, 4, 151936, 0.3), (4, 2, 8, 151936, 0.3), (3, 5, 3, 4096, 0.3), (2, 64, 1, 300, 0.3),
         (5, 3, 6, 9000, 0.3), (2, 7, 0, 1000, 0.3), (16, 4, 4, 2000, 2.0), (8, 8, 3, 151936, 1.5)]


@pytest.mark.parametrize("b,c,kd,v,noise", CASES)
def test_multi_accept_matches_the_oracle(b, c, kd, v, noise):
    dl, tl, tok, u = make_case(b, c, kd, v, seed=b * 1000 + c * 10 + kd, noise=noise)
    q_out = torch.empty((kd, b, c, v), device=DEV)
    p_out = torch.empty((b, c, kd + 1, v), device=DEV)
    n, t, ch = sq.sq_spec_accept_multi(dl.to(DEV) if kd else None, tl.to(DEV), tok.to(DEV) if kd else None,
                                       u.to(DEV), 1.0, q_out=q_out if kd else None, p_out=p_out)
    torch.cuda.synchronize()
    n, t, ch = n.cpu().numpy(), t.cpu().numpy(), ch.cpu().numpy()
    u32 = u.numpy().view(np.uint32)
    # the rule on the kernel's own fp32 distributions: bit for bit
    q32 = q_out.cpu().numpy() if kd else None
    n_o, t_o, ch_o = oracle.multi_accept_probs(p_out.cpu().numpy(), q32, tok.numpy() if kd else None, u32)
    assert np.array_equal(n, n_o) and np.array_equal(t, t_o) and np.array_equal(ch, ch_o)
    # the distributions: the oracle's fp64 softmax, rounded to fp32 (or one ulp from it)
    pref = oracle.softmax(tl.reshape(-1, v).numpy()).reshape(b, c, kd + 1, v)
    p32 = p_out.cpu().numpy()
    assert (np.abs(p32 - pref) <= np.spacing(pref.astype(np.float32)) * 1.01).all()
    # end to end from the logits
    n_e, t_e, ch_e = oracle.multi_accept(dl.numpy() if kd else None, tl.numpy(), tok.numpy() if kd else None, u32,
                                         1.0)
    same = (n_e == n) & (t_e == t) & (ch_e == ch)
    assert same.mean() >= 0.99 and (n >= 0).all() and (t >= 0).all()
    if kd:
        assert 0 <= n.min() and n.max() <= kd
    print(f"\n[multi] b {b} c {c} kd {kd} v {v}: n {n.tolist()} chains {ch.tolist()}", flush=True)


def test_one_chain_equals_the_single_candidate_call():
    b, kd, v = 6, 5, 20000
    dl, tl, tok, u = make_case(b, 1, kd, v, seed=77)
    n1, t1 = sq.sq_spec_accept(dl.reshape(kd, b, v).to(DEV), tl.reshape(b, kd + 1, v).to(DEV),
                               tok.reshape(kd, b).to(DEV), u.to(DEV), 1.0)
    n2, t2, ch = sq.sq_spec_accept_multi(dl.to(DEV), tl.to(DEV), tok.to(DEV), u.to(DEV), 1.0)
    torch.cuda.synchronize()
    assert torch.equal(n1, n2) and torch.equal(t1, t2) and (ch == 0).all()
    assert len(set(n1.tolist())) > 1


def test_multi_greedy_and_rows_without_a_distribution():
    b, c, kd, v = 4, 3, 3, 5000
    dl, tl, tok, u = make_case(b, c, kd, v, seed=5)
    # make chains follow the argmax for a while: chain 1 of sequence 0 takes it at every depth
    for d in range(kd):
        tok[d, 0, 1] = int(torch.argmax(tl[0, 1, d]))
    tl[0, 0] = tl[0, 1]  # the lowest alive chain's rows are the ones read
    n, t, ch = sq.sq_spec_accept_multi(dl.to(DEV), tl.to(DEV), tok.to(DEV), None, 0.0)
    torch.cuda.synchronize()
    n_o, t_o, ch_o = oracle.multi_accept_greedy(tl.numpy(), tok.numpy())
    assert np.array_equal(n.cpu().numpy(), n_o) and np.array_equal(t.cpu().numpy(), t_o)
    assert np.array_equal(ch.cpu().numpy(), ch_o) and n_o[0] == kd
    # a NaN in one row of sequence 2 (T > 0) and a +inf in sequence 3 (T = 0)
    tl2 = tl.clone()
    tl2[2, 1, 2, 17] = float("nan")
    n, t, ch = sq.sq_spec_accept_multi(dl.to(DEV), tl2.to(DEV), tok.to(DEV), u.to(DEV), 1.0)
    torch.cuda.synchronize()
    assert n[2].item() == t[2].item() == ch[2].item() == -1 and (n[[0, 1, 3]] >= 0).all()
    tl2 = tl.clone()
    tl2[3, 2, 0, 5] = float("inf")
    n, t, ch = sq.sq_spec_accept_multi(dl.to(DEV), tl2.to(DEV), tok.to(DEV), None, 0.0)
    torch.cuda.synchronize()
    assert n[3].item() == t[3].item() == ch[3].item() == -1 and (n[:3] >= 0).all()


def test_kv_adopt_and_commit_multi():
    layers, b, c, hkv, cap, kd = 3, 2, 3, 2, 128, 4
    g = gen(3)
    kc = torch.randn((layers, b * c, hkv, cap, 128), generator=g).half().to(DEV)
    vc = torch.randn((layers, b * c, hkv, 128, cap), generator=g).half().to(DEV)
    k0, v0 = kc.clone(), vc.clone()
    chain = torch.tensor([2, 0], dtype=torch.int32, device=DEV)
    n = torch.tensor([3, 0], dtype=torch.int32, device=DEV)
    pos = torch.tensor([50, 50, 50, 70, 70, 70], dtype=torch.int32, device=DEV)
    sq.sq_kv_adopt_f16(kc, vc, b, c, chain, n, pos, -1, 0)
    torch.cuda.synchronize()
    for s, src, lo, hi in ((0, 2, 49, 53), (1, 0, 69, 70)):
        for j in range(c):
            r = s * c + j
            exp_k, exp_v = k0[:, r].clone(), v0[:, r].clone()
            if j != src:
                exp_k[:, :, lo:hi + 1] = k0[:, s * c + src, :, lo:hi + 1]
                exp_v[:, :, :, lo:hi + 1] = v0[:, s * c + src, :, :, lo:hi + 1]
            assert torch.equal(kc[:, r], exp_k) and torch.equal(vc[:, r], exp_v)
    # commit: sequence 0 accepted 3 drafts of chain 2, sequence 1 none
    drafts = torch.arange(kd * b * c, dtype=torch.int32, device=DEV).view(kd, b * c)
    nxt = torch.tensor([900, 901], dtype=torch.int32, device=DEV)
    pending = torch.tensor([7, 7, 7, 8, 8, 8], dtype=torch.int32, device=DEV)
    prev = torch.zeros(6, dtype=torch.int32, device=DEV)
    out = torch.full((b, 8), -1, dtype=torch.int32, device=DEV)
    out_len = torch.zeros(b, dtype=torch.int32, device=DEV)
    status = torch.zeros(1, dtype=torch.int32, device=DEV)
    sq.sq_spec_commit_multi(n, nxt, chain, drafts, c, pending, prev, pos, out_tokens=out, out_len=out_len,
                            status=status)
    torch.cuda.synchronize()
    d = drafts.view(kd, b, c).cpu()
    assert out[0, :4].tolist() == [int(d[0, 0, 2]), int(d[1, 0, 2]), int(d[2, 0, 2]), 900]
    assert out[1, :1].tolist() == [901] and out_len.tolist() == [4, 1]
    assert pending.tolist() == [900] * 3 + [901] * 3
    assert prev.tolist() == [int(d[2, 0, 2])] * 3 + [8] * 3
    assert pos.tolist() == [54] * 3 + [71] * 3 and status.item() == 0
