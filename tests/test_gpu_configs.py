"""GPU parity at the five workloads' full shapes, through the resident stack and
round driver that the benchmark times, against the CPU oracle.

Workload 0 (one Qwen2.5-0.5B-shaped layer) is checked in full.  Workloads 1-4
build every layer:
  - quantized codes bit for bit: every row of every matrix for workloads 1
    and 2; for workloads 3 and 4 every row of layers 0 and L-1 and the LM
    head, and 1 % of the rows (at least 64, plus the first and last) of every
    other matrix;
  - the draft GEMV and the verify GEMM within the normalised-error bound: every
    row of layers 0 and L-1 and the LM head, 64 seeded rows (plus the first
    and last) of every other matrix.  At 36 verify rows (workload 3) the fp64
    oracle GEMM over whole matrices would take minutes, so there the verify
    GEMM is checked on 256 seeded rows of every matrix.
Two whole rounds then run through the driver.  Their draft draws and accept
steps are checked bit for bit against the oracle run on the kernels' own fp32
distributions, and end to end against the oracle's own softmax of the
rounds' logits up to counted near-ties (none expected)."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_21704_amd as sq
from paper_2609_21704_amd import synth
from paper_2609_21704_amd.configs import CONFIGS
from paper_2609_21704_amd.rounds import DirectDecode, Round, Stack, round_uniforms
from accept_compare import check_accept

pytestmark = pytest.mark.gpu
DEV = "cuda"
GEMV_TOL = 2e-3


def bits16(t: torch.Tensor) -> np.ndarray:
    return t.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)


def sample_rows(n: int, seed: int, count: int = 64) -> np.ndarray:
    g = torch.Generator().manual_seed(seed)
    rows = torch.randperm(n, generator=g)[:count].numpy()
    return np.unique(np.concatenate([rows, [0, n - 1]]))


def check_quant(stack: Stack, key, rows):
    """The draft copy's codes, scales (and zeros) at `rows`, bit for bit."""
    w16 = stack.w16[key]
    idx = torch.from_numpy(rows).to(DEV)
    w_rows = bits16(w16.index_select(0, idx))
    pack = stack.draft[key]
    if stack.variant == "int4":
        ref = oracle.quantize_int4_g128(w_rows)
        assert np.array_equal(pack[0].index_select(0, idx).cpu().numpy(), ref[0]), key
        assert np.array_equal(bits16(pack[1].index_select(0, idx)), ref[1]), key
        assert np.array_equal(bits16(pack[2].index_select(0, idx)), ref[2]), key
    else:
        ref = oracle.quantize_fp8_e4m3(w_rows)
        assert np.array_equal(pack[0].index_select(0, idx).cpu().numpy(), ref[0]), key
        assert np.array_equal(pack[1].index_select(0, idx).cpu().numpy().view(np.uint32), ref[1].view(np.uint32)), key
    return w_rows, ref


def check_products(stack: Stack, key, rows, seed: int, w_rows=None, ref=None, draft=True, verify=True):
    """The draft GEMV (m = B) and the verify GEMM (m = B(k+1)) at `rows`, with
    the output types the driver uses."""
    cfg = stack.cfg
    if w_rows is None:
        w_rows, ref = check_quant(stack, key, rows)
    n, k = stack.w16[key].shape
    idx = torch.from_numpy(rows).to(DEV)
    y_dtype = torch.float32 if key[1] == "lm_head" else torch.float16
    if draft:
        check_draft(stack, key, idx, seed, ref, y_dtype)
    if not verify:
        return
    xv = synth.normal_f16((cfg.verify_m, k), 1.0, synth.stream_seed(seed, 2), DEV)
    yv = torch.empty((cfg.verify_m, n), dtype=y_dtype, device=DEV)
    stack.verify_gemm(key, xv, yv)
    yv_ref, dv_ref = oracle.gemm_f16(bits16(xv), w_rows)
    err = oracle.normalised_error(yv.index_select(1, idx).float().cpu().numpy(), yv_ref, dv_ref)
    assert err <= GEMV_TOL, (key, "verify", err)


def check_draft(stack: Stack, key, idx, seed: int, ref, y_dtype):
    cfg = stack.cfg
    n, k = stack.w16[key].shape
    xd = synth.normal_f16((cfg.draft_m, k), 1.0, synth.stream_seed(seed, 1), DEV)
    y = torch.empty((cfg.draft_m, n), dtype=y_dtype, device=DEV)
    stack.draft_gemv(key, xd, y)
    if stack.variant == "int4":
        y_ref, d_ref = oracle.qgemv_w4a16(bits16(xd), *ref)
    else:
        y_ref, d_ref = oracle.qgemv_w8a16(bits16(xd), *ref)
    err = oracle.normalised_error(y.index_select(1, idx).float().cpu().numpy(), y_ref, d_ref)
    assert err <= GEMV_TOL, (key, "draft", err)


def check_matrix(stack: Stack, key, rows, seed: int):
    """Quantized rows bit for bit, then the draft GEMV and verify GEMM at those rows."""
    w_rows, ref = check_quant(stack, key, rows)
    check_products(stack, key, rows, seed, w_rows, ref)


def check_round(rnd: Round, round_index: int):
    """Run one round and check its draws and accept step against the oracle."""
    cfg = rnd.cfg
    B, k, V = cfg.batch, cfg.k, cfg.vocab
    T = rnd.temperature
    ud, ua = round_uniforms(cfg, round_index + 1, DEV)
    rnd.set_uniforms(ud[round_index], ua[round_index])
    rnd.run()
    torch.cuda.synchronize()
    b = rnd.buf
    draft = b.draft_logits.cpu().numpy()
    target = b.target_logits.cpu().numpy()
    tokens = b.draft_tokens.cpu().numpy()
    u_d = b.u_draft.cpu().numpy().view(np.uint32)
    u_a = b.u_accept.cpu().numpy().view(np.uint32)
    dev = b.n_accepted.device
    for i in range(k):  # draft draw i: a plain sampler over draft row i
        if T > 0:
            p_i = torch.empty((B, 1, V), dtype=torch.float32, device=dev)
            n_i, t_i = sq.sq_spec_accept(None, b.draft_logits[i].view(B, 1, V), None, b.u_draft[i].view(B, 1), T,
                                         p_out=p_i)
            assert np.array_equal(t_i.cpu().numpy(), tokens[i]), ("draft draw", i)
            check_accept(None, draft[i].reshape(B, 1, V), np.zeros((0, B), np.int32), u_d[i].reshape(B, 1), T,
                         n_i.cpu().numpy(), tokens[i], None, p_i.cpu().numpy())
        else:
            check_accept(None, draft[i].reshape(B, 1, V), np.zeros((0, B), np.int32), None, T,
                         np.zeros(B, np.int32), tokens[i])
    n_gpu, t_gpu = b.n_accepted.cpu().numpy(), b.next_token.cpu().numpy()
    if T > 0:  # the accept step again with its distributions, to check it on the kernel's own p / q
        q_o = torch.empty((k, B, V), dtype=torch.float32, device=dev)
        p_o = torch.empty((B, k + 1, V), dtype=torch.float32, device=dev)
        n2, t2 = sq.sq_spec_accept(b.draft_logits, b.target_logits, b.draft_tokens, b.u_accept, T, q_out=q_o,
                                   p_out=p_o)
        assert np.array_equal(n2.cpu().numpy(), n_gpu) and np.array_equal(t2.cpu().numpy(), t_gpu)
        check_accept(draft, target, tokens, u_a, T, n_gpu, t_gpu, q_o.cpu().numpy(), p_o.cpu().numpy())
    else:
        check_accept(draft, target, tokens, None, T, n_gpu, t_gpu)
    return n_gpu


@pytest.mark.parametrize("variant", ["int4", "fp8"])
def test_workload0_full(variant):
    cfg = CONFIGS[0]
    stack = Stack(cfg, DEV, variant=variant)
    for key in stack.w16:
        n = stack.w16[key].shape[0]
        check_matrix(stack, key, np.arange(n), seed=cfg.seed * 100 + len(key[1]))
    rnd = Round(stack, temperature=1.0)
    for r in range(3):
        check_round(rnd, r)
    greedy = Round(stack, temperature=0.0)
    check_round(greedy, 0)


WORKLOADS = [(1, "int4"), (1, "fp8"), (2, "int4"), (3, "fp8"), (4, "int4")]


@pytest.mark.parametrize("index,variant", WORKLOADS)
def test_workload_whole_stack(index, variant):
    cfg = CONFIGS[index]
    stack = Stack(cfg, DEV, variant=variant)
    last = cfg.layers - 1
    all_codes = index in (1, 2)  # every row's codes for the 1.5B and 7B stacks
    for j, key in enumerate(sorted(stack.w16)):
        n = stack.w16[key].shape[0]
        full = key[0] in (0, last) or key[1] == "lm_head"
        seed = cfg.seed * 100 + j
        if full and cfg.verify_m <= 8:
            check_matrix(stack, key, np.arange(n), seed)
            continue
        if full:  # codes and the draft GEMV on every row, the verify GEMM on sampled rows
            w_rows, ref = check_quant(stack, key, np.arange(n))
            check_products(stack, key, np.arange(n), seed, w_rows, ref, verify=False)
            check_products(stack, key, sample_rows(n, cfg.seed * 3000 + j, count=256), seed, draft=False)
            continue
        prod_rows = sample_rows(n, cfg.seed * 1000 + j)
        if all_codes:
            check_quant(stack, key, np.arange(n))
            check_products(stack, key, prod_rows, seed)
        else:
            check_quant(stack, key, sample_rows(n, cfg.seed * 2000 + j, count=max(64, n // 100)))
            check_products(stack, key, prod_rows, seed)
    rnd = Round(stack, temperature=1.0)
    check_round(rnd, 0)
    check_round(rnd, 1)
    del rnd, stack
    torch.cuda.empty_cache()


def test_round_graph_replays_match_eager():
    """One round captured as a HIP graph: each replay (fresh uniforms, eager
    work and synchronisations in between) gives the eager round's bits."""
    cfg = CONFIGS[0]
    stack = Stack(cfg, DEV)
    rnd = Round(stack, temperature=1.0)
    rnd.capture()
    ud, ua = round_uniforms(cfg, 4, DEV)
    for r in range(4):
        rnd.set_uniforms(ud[r], ua[r])
        rnd.replay()
        torch.cuda.synchronize()
        b = rnd.buf
        got = [t.clone() for t in (b.draft_logits, b.target_logits, b.draft_tokens, b.n_accepted, b.next_token)]
        rnd.set_uniforms(ud[r], ua[r])
        rnd.run()
        torch.cuda.synchronize()
        ref = (b.draft_logits, b.target_logits, b.draft_tokens, b.n_accepted, b.next_token)
        for g, e in zip(got, ref):
            assert torch.equal(g, e), r


@pytest.mark.parametrize("index", [0, 1])
def test_direct_decode_matches_oracle(index):
    """Direct parent inference (the plain-decoding baseline): every FP16
    projection at m = batch, then the draw, against the oracle at sampled
    rows; captured as a HIP graph, the replays give the eager step's bits."""
    cfg = CONFIGS[index]
    stack = Stack(cfg, DEV, layers=1)
    dd = DirectDecode(stack, temperature=1.0)
    dd.u.copy_(synth.uniform_u24((cfg.batch, 1), 77, DEV))
    dd.run()
    torch.cuda.synchronize()
    for j, key in enumerate(sorted(k for k in stack.w16 if k[1] != "lm_head")):
        w16 = stack.w16[key]
        rows = sample_rows(w16.shape[0], cfg.seed * 10 + j)
        idx = torch.from_numpy(rows).to(DEV)
        y_ref, d_ref = oracle.gemm_f16(bits16(dd.x[key]), bits16(w16.index_select(0, idx)))
        err = oracle.normalised_error(dd.y[key[1]].index_select(1, idx).float().cpu().numpy(), y_ref, d_ref)
        assert err <= GEMV_TOL, (key, err)
    if cfg.lm_head:
        key = (cfg.layers, "lm_head")
        rows = sample_rows(cfg.vocab, cfg.seed * 10 + 9)
        idx = torch.from_numpy(rows).to(DEV)
        y_ref, d_ref = oracle.gemm_f16(bits16(dd.x[(stack.layers, "lm_head")]), bits16(stack.w16[key].index_select(0, idx)))
        err = oracle.normalised_error(dd.logits.index_select(1, idx).cpu().numpy(), y_ref, d_ref)
        assert err <= GEMV_TOL, err
    B, V = cfg.batch, cfg.vocab
    logits = dd.logits.cpu().numpy().reshape(B, 1, V)
    p_o = torch.empty((B, 1, V), dtype=torch.float32, device=DEV)   # the same draw again, with its distribution
    n2, t2 = sq.sq_spec_accept(None, dd.logits.view(B, 1, V), None, dd.u, 1.0, p_out=p_o)
    assert torch.equal(t2, dd.token) and torch.equal(n2, dd.n_accepted)
    check_accept(None, logits, np.zeros((0, B), np.int32), dd.u.cpu().numpy(), 1.0, dd.n_accepted.cpu().numpy(),
                 dd.token.cpu().numpy(), None, p_o.cpu().numpy())
    eager = dd.token.clone()
    dd.capture()
    for _ in range(3):
        dd.replay()
        torch.cuda.synchronize()
        assert torch.equal(dd.token, eager)
    del dd, stack
    torch.cuda.empty_cache()


def test_round_acceptance_law_from_its_own_distributions():
    """Over 4000 rounds of workload 0 (its draft and parent rows are the same
    every round; only the uniforms change), n_accepted follows the closed form
    P(n = i) = prod_{j<i} beta_j (1 - beta_i), P(n = k) = prod beta, with
    beta_j = sum_x min(p_j(x), q_j(x)) from the round's own distributions, and
    the mean tokens per round (n + 1) is within sampling error of
    1 + sum_{i=1..k} prod_{j<i} beta_j, the figure the benchmark reports."""
    from scipy import stats

    cfg = CONFIGS[0]
    B, k, V = cfg.batch, cfg.k, cfg.vocab
    stack = Stack(cfg, DEV)
    rnd = Round(stack, temperature=1.0)
    R = 4000
    ud, ua = round_uniforms(cfg, R, DEV)
    rnd.set_uniforms(ud[0], ua[0])
    rnd.capture()
    n_hist = torch.empty((R, B), dtype=torch.int32, device=DEV)
    for r in range(R):
        rnd.set_uniforms(ud[r], ua[r])
        rnd.replay()
        n_hist[r].copy_(rnd.buf.n_accepted)
    torch.cuda.synchronize()
    b = rnd.buf
    q = torch.empty((k, B, V), dtype=torch.float32, device=DEV)
    p = torch.empty((B, k + 1, V), dtype=torch.float32, device=DEV)
    sq.sq_spec_accept(b.draft_logits, b.target_logits, b.draft_tokens, b.u_accept, 1.0, q_out=q, p_out=p)
    pn, qn = p.cpu().numpy().astype(np.float64), q.cpu().numpy().astype(np.float64)
    beta = np.minimum(pn[0, :k], qn[:, 0]).sum(axis=1)
    law = np.array([np.prod(beta[:i]) * (1 - beta[i]) for i in range(k)] + [np.prod(beta)])
    assert abs(law.sum() - 1) < 1e-12
    n = n_hist.cpu().numpy().ravel()
    obs = np.bincount(n, minlength=k + 1)
    chi2 = np.sum((obs - n.size * law) ** 2 / (n.size * law))
    assert chi2 < stats.chi2.ppf(1 - 1e-3, k), (chi2, obs, n.size * law)
    expected = 1.0 + np.cumprod(beta).sum()
    assert abs(expected - (np.arange(k + 1) + 1) @ law) < 1e-12
    sd = np.sqrt(((np.arange(k + 1) + 1) ** 2) @ law - expected ** 2)
    assert abs((n + 1).mean() - expected) < 4 * sd / np.sqrt(n.size), ((n + 1).mean(), expected)
