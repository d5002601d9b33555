"""GPU checks of the decoder's fused projections: a projection that
normalises its own input rows (sq_qgemv_w4a16_rmsnorm,
sq_verify_gemm_f16_rmsnorm) must give the bits of sq_add_rmsnorm_f16
followed by the plain projection, and a projection added into the residual
stream (sq_qgemv_w4a16_acc, sq_verify_gemm_f16_acc) the bits of the plain
projection followed by one fp32 add, the gate|up projection with the SiLU
product in its epilogue the bits of the three calls, and the attention that
rotates its own rows (sq_rope_attention_f16) the bits of sq_rope_kv_f16 +
sq_attention_f16 (output, both caches, status); shapes without a fused
kernel return False and leave the output untouched.  Rounds through the decoder with and
without the fused forms are then equal bit for bit (tokens, positions,
caches, logits).  The unfused calls are themselves checked against the
oracle in test_gpu_decoder.py and test_gpu_parity.py."""
import pytest
import torch

import paper_2609_21704_amd as sq
from paper_2609_21704_amd import decoder as dec
from paper_2609_21704_amd import synth
from paper_2609_21704_amd.configs import CONFIGS

pytestmark = pytest.mark.gpu
DEV = "cuda"
EPS = 1e-6


def gen(seed):
    g = torch.Generator(device="cpu")
    g.manual_seed(seed)
    return g


def bits(t):
    return t.contiguous().view(torch.int32 if t.dtype == torch.float32 else torch.int16)


def int4_weights(n, k, seed):
    w = (torch.randn((n, k), generator=gen(seed)) * 0.02).half().to(DEV)
    return sq.sq_quantize_int4_g128(w)


def residual(mg, k, seed, scale=3.0):
    g = gen(seed)
    h = (torch.randn((mg, k), generator=g) * scale).float().to(DEV)
    nw = (1.0 + torch.randn((k,), generator=g) * 0.02).half().to(DEV)
    return h, nw


# draft (INT4) shapes: row blocks (q|k|v, o, 1.5B), tasks of rows (gate|up, LM head)
W4_NORM = [(4608, 3584, 1, 1), (4608, 3584, 2, 1), (37888, 3584, 1, 1), (37888, 3584, 2, 1),
           (151936, 3584, 1, 2), (151936, 3584, 1, 1), (2048, 1536, 2, 1), (17920, 1536, 1, 1), (4608, 3584, 1, 5)]


@pytest.mark.parametrize("n,k,m,group", W4_NORM)
def test_qgemv_w4a16_rmsnorm_equals_norm_then_gemv(n, k, m, group):
    codes, scales, zeros = int4_weights(n, k, n + k)
    h, nw = residual(m * group, k, n + m)
    h0 = h.clone()
    y = torch.full((m, n), float("nan"), device=DEV)
    assert sq.sq_qgemv_w4a16_rmsnorm(h, nw, EPS, codes, scales, zeros, group=group, y=y)
    x = sq.sq_add_rmsnorm_f16(h.clone(), nw, EPS, group=group)
    ref = sq.sq_qgemv_w4a16(x, codes, scales, zeros)
    torch.cuda.synchronize()
    assert torch.equal(h, h0)
    assert torch.equal(bits(y), bits(ref))


@pytest.mark.parametrize("n,k,m", [(4608, 3584, 5), (3584, 3584, 5), (4864, 896, 5), (2048, 1536, 8),
                                   (4608, 3584, 1)])
def test_verify_gemm_f16_rmsnorm_equals_norm_then_gemm(n, k, m):
    w16 = (torch.randn((n, k), generator=gen(n)) * 0.02).half().to(DEV)
    h, nw = residual(m, k, n + 7)
    y = torch.empty((m, n), device=DEV)
    assert sq.sq_verify_gemm_f16_rmsnorm(h, nw, EPS, w16, y=y)
    x = sq.sq_add_rmsnorm_f16(h.clone(), nw, EPS)
    ref = sq.sq_verify_gemm_f16(x, w16)
    torch.cuda.synchronize()
    assert torch.equal(bits(y), bits(ref))


@pytest.mark.parametrize("n,k,m,group", [(37888, 3584, 1, 1), (37888, 3584, 2, 1), (37888, 3584, 1, 3),
                                         (55296, 3584, 1, 1), (36864, 4096, 2, 1)])
def test_qgemv_w4a16_rmsnorm_silu_equals_three_calls(n, k, m, group):
    codes, scales, zeros = int4_weights(n, k, n + 2 * k)
    h, nw = residual(m * group, k, n + 3)
    t = torch.full((m, n // 2), float("nan"), dtype=torch.float16, device=DEV)
    assert sq.sq_qgemv_w4a16_rmsnorm_silu(h, nw, EPS, codes, scales, zeros, t, group=group)
    x = sq.sq_add_rmsnorm_f16(h.clone(), nw, EPS, group=group)
    gu = sq.sq_qgemv_w4a16(x, codes, scales, zeros)
    ref = sq.sq_silu_mul_f16(gu)
    torch.cuda.synchronize()
    assert torch.equal(bits(t), bits(ref))


def test_silu_fusion_unsupported_shapes_enqueue_nothing():
    codes, scales, zeros = int4_weights(4096, 3584, 11)  # 2048 gate rows: fewer tasks than wavefronts
    h, nw = residual(1, 3584, 12)
    t = torch.full((1, 2048), 7.0, dtype=torch.float16, device=DEV)
    assert not sq.sq_qgemv_w4a16_rmsnorm_silu(h, nw, EPS, codes, scales, zeros, t)
    c1, s1, z1 = int4_weights(17920, 1536, 15)  # rows of 1536 k: the plain projection takes the row blocks
    h1, nw1 = residual(1, 1536, 16)
    t1 = torch.full((1, 8960), 7.0, dtype=torch.float16, device=DEV)
    assert not sq.sq_qgemv_w4a16_rmsnorm_silu(h1, nw1, EPS, c1, s1, z1, t1)
    c2, s2, z2 = int4_weights(37888, 3584, 13)
    h3, nw3 = residual(3, 3584, 14)
    t3 = torch.full((3, 18944), 7.0, dtype=torch.float16, device=DEV)
    assert not sq.sq_qgemv_w4a16_rmsnorm_silu(h3, nw3, EPS, c2, s2, z2, t3)  # m = 3
    torch.cuda.synchronize()
    assert (t == 7.0).all() and (t3 == 7.0).all() and (t1 == 7.0).all()


def test_fused_norm_unsupported_shapes_enqueue_nothing():
    codes, scales, zeros = int4_weights(4608, 3584, 3)
    h, nw = residual(3, 3584, 4)
    y = torch.full((3, 4608), 7.0, device=DEV)
    assert not sq.sq_qgemv_w4a16_rmsnorm(h, nw, EPS, codes, scales, zeros, y=y)  # m = 3: no fused kernel
    w16 = (torch.randn((37888, 3584), generator=gen(5)) * 0.02).half().to(DEV)
    h5, _ = residual(5, 3584, 6)
    y5 = torch.full((5, 37888), 7.0, device=DEV)
    assert not sq.sq_verify_gemm_f16_rmsnorm(h5, nw, EPS, w16, y=y5)  # beyond the row-block kernel
    hk, nwk = residual(1, 5120, 8)
    c2, s2, z2 = int4_weights(5120, 5120, 9)
    yk = torch.full((1, 5120), 7.0, device=DEV)
    assert not sq.sq_qgemv_w4a16_rmsnorm(hk, nwk, EPS, c2, s2, z2, y=yk)  # rows longer than 4096
    torch.cuda.synchronize()
    assert (y == 7.0).all() and (y5 == 7.0).all() and (yk == 7.0).all()


@pytest.mark.parametrize("n,k,m", [(3584, 3584, 1), (3584, 18944, 1), (3584, 18944, 2), (1536, 8960, 1),
                                   (37888, 3584, 1), (4608, 3584, 4)])
def test_qgemv_w4a16_acc_equals_gemv_then_add(n, k, m):
    codes, scales, zeros = int4_weights(n, k, n * 3 + k)
    x = torch.randn((m, k), generator=gen(k)).half().to(DEV)
    y0 = (torch.randn((m, n), generator=gen(n)) * 5).float().to(DEV)
    y = y0.clone()
    assert sq.sq_qgemv_w4a16_acc(x, codes, scales, zeros, y)
    p = sq.sq_qgemv_w4a16(x, codes, scales, zeros)
    torch.cuda.synchronize()
    assert torch.equal(bits(y), bits(y0 + p))


@pytest.mark.parametrize("n,k,m", [(3584, 3584, 5), (3584, 18944, 5), (1536, 8960, 8), (4608, 3584, 1)])
def test_verify_gemm_f16_acc_equals_gemm_then_add(n, k, m):
    w16 = (torch.randn((n, k), generator=gen(n + 1)) * 0.02).half().to(DEV)
    x = torch.randn((m, k), generator=gen(k + 1)).half().to(DEV)
    y0 = (torch.randn((m, n), generator=gen(m)) * 5).float().to(DEV)
    y = y0.clone()
    assert sq.sq_verify_gemm_f16_acc(x, w16, y)
    p = sq.sq_verify_gemm_f16(x, w16)
    # a second call on the same K-slice meeting slots: they were left empty
    y2 = y0.clone()
    assert sq.sq_verify_gemm_f16_acc(x, w16, y2)
    torch.cuda.synchronize()
    assert torch.equal(bits(y), bits(y0 + p)) and torch.equal(bits(y2), bits(y))


@pytest.mark.parametrize("ci,layers,B,k,chains", [(2, 2, 1, 4, 1), (1, 2, 2, 3, 1), (1, 2, 1, 2, 2)])
def test_fused_rounds_equal_unfused_rounds(ci, layers, B, k, chains):
    """Decoder rounds with the fused projections reproduce the unfused rounds
    bit for bit: tokens, positions, both caches and the last logits."""
    cfg = CONFIGS[ci]
    w = dec.DecoderWeights(cfg, DEV, layers=layers)
    cap, R = 256, 3
    runs = []
    for fuse in (True, False):
        sd = dec.SpecDecoder(w, batch=B, k=k, capacity=cap, chains=chains, fuse=fuse)
        sd.prefill(dec.synthetic_prompt(cfg, B, 40, DEV))
        ud = synth.uniform_u24((R, k, B * chains), synth.stream_seed(cfg.seed, 97), DEV)
        ua = synth.uniform_u24((R, B, chains * k + 1), synth.stream_seed(cfg.seed, 98), DEV)
        for r in range(R):
            sd.set_uniforms(ud[r], ua[r])
            sd.run()
        torch.cuda.synchronize()
        assert sd.status.item() == 0
        runs.append((sd.out_tokens[:, :int(sd.out_len.max())].clone(), sd.pos_base.clone(),
                     sd.target_logits.clone(), sd.draft_logits.clone(), sd.pcache.k_all.clone(),
                     sd.pcache.v_all.clone(), sd.dcache.k_all.clone(), sd.dcache.v_all.clone()))
        del sd
    for a, b, what in zip(runs[0], runs[1], ("tokens", "positions", "target logits", "draft logits", "parent keys",
                                              "parent values", "draft keys", "draft values")):
        assert torch.equal(bits(a) if a.is_floating_point() else a, bits(b) if b.is_floating_point() else b), what


def rope_block(b, rps, hq, hkv, cap, pb, seed, with_bias=True):
    """Projection rows, bias and caches full of finite stale entries."""
    g = gen(seed)
    nh = hq + 2 * hkv
    qkv = (torch.randn((b * rps, nh * 128), generator=g) * 2).float().to(DEV)
    bias = (torch.randn((nh * 128,), generator=g) * 0.5).half().to(DEV) if with_bias else None
    kc = (torch.randn((b, hkv, cap, 128), generator=g)).half().to(DEV)
    vc = (torch.randn((b, hkv, 128, cap), generator=g)).half().to(DEV)
    return qkv, bias, kc, vc, torch.tensor(pb, dtype=torch.int32, device=DEV)


# (b, rps, hq, hkv, capacity, len_bound, pos_base, offset, bias): the 7B draft
# step and verification block (a block across a chunk boundary), four
# sequences of 9 rows (four query tiles), a long cache (slots of several
# chunks), the 1.5B heads without bias, one query head per kv head with 16
# rows from position 0, rows before 0 and past len_bound (a sequence with
# every row before 0 among them), and one query tile over 64 slots
ROPE_ATT = [(1, 1, 28, 4, 2048, 2048, [1100], 0, True),
            (1, 5, 28, 4, 2048, 2048, [1020], 2, True),
            (4, 9, 28, 4, 4096, 4096, [100, 1000, 2040, 4000], 0, True),
            (4, 9, 28, 4, 8192, 8192, [8000, 7000, 64, 8180], 1, True),
            (2, 5, 12, 2, 1024, 1024, [511, 0], 0, False),
            (1, 16, 8, 8, 512, 512, [0], 0, True),
            (3, 5, 28, 4, 1024, 900, [-3, 897, 60], 0, True),
            (2, 1, 28, 4, 1024, 900, [-5, 100], 0, True),
            (1, 2, 14, 2, 1024, 512, [511], 0, True),
            (1, 1, 28, 4, 4096, 4096, [3000], 0, True)]


@pytest.mark.parametrize("b,rps,hq,hkv,cap,lb,pb,off,with_bias", ROPE_ATT)
def test_rope_attention_equals_rope_then_attention(b, rps, hq, hkv, cap, lb, pb, off, with_bias):
    qkv, bias, kc, vc, pbt = rope_block(b, rps, hq, hkv, cap, pb, 500 + rps + cap, with_bias)
    k1, v1, k2, v2 = kc.clone(), vc.clone(), kc.clone(), vc.clone()
    s1 = torch.zeros(1, dtype=torch.int32, device=DEV)
    s2 = torch.zeros(1, dtype=torch.int32, device=DEV)
    q = sq.sq_rope_kv_f16(qkv, bias, pbt, off, rps, hq, k1, v1, len_bound=lb, theta=1e6, status=s1)
    out1 = sq.sq_attention_f16(q, k1, v1, pbt, off, rps, len_bound=lb)
    out2 = torch.full_like(out1, 7.0)
    assert sq.sq_rope_attention_f16(qkv, bias, pbt, off, rps, hq, k2, v2, out2, len_bound=lb, theta=1e6, status=s2)
    torch.cuda.synchronize()
    assert torch.equal(bits(out1), bits(out2))
    assert torch.equal(bits(k1), bits(k2)) and torch.equal(bits(v1), bits(v2))
    assert int(s1.item()) == int(s2.item())
    bad = any(p + off + j < 0 or p + off + j >= lb for p in pb for j in range(rps))
    assert (int(s2.item()) != 0) == bad


def test_rope_attention_unsupported_blocks_enqueue_nothing():
    for b, rps, hq, hkv in ((1, 17, 8, 8), (1, 10, 28, 4)):
        qkv, bias, kc, vc, pbt = rope_block(b, rps, hq, hkv, 1024, [100] * b, 77)
        k0, v0 = kc.clone(), vc.clone()
        out = torch.full((b * rps, hq, 128), 3.0, dtype=torch.float16, device=DEV)
        assert not sq.sq_rope_attention_f16(qkv, bias, pbt, 0, rps, hq, kc, vc, out)
        torch.cuda.synchronize()
        assert torch.equal(kc, k0) and torch.equal(vc, v0) and bool((out == 3.0).all())
