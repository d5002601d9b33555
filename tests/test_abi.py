"""CPU-only checks of the C ABI: the built library loads, exports every symbol
the header declares, and rejects invalid arguments on the host before any HIP
call (fake, never dereferenced device addresses are passed)."""
import os
import re

import pytest

import paper_2609_21704_amd as sq

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "specquant.h")

OK, NULL, SHAPE, ALIGN, ALIAS, NONFINITE, UNSUPPORTED, DEVICE, CAPTURE = 0, 1, 2, 3, 4, 5, 6, 7, 8
A = 0x7F0000000000          # 16-byte aligned fake addresses, far apart
B = A + (1 << 32)
C = A + (2 << 32)
D = A + (3 << 32)
E = A + (4 << 32)
F32, F16 = 1, 0


def declared_symbols():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:sq_status|const char\*|int32_t)\s+(sq_\w+)\s*\(", text, re.M)))


def test_library_exports_every_declared_symbol():
    lib = sq.load()
    names = declared_symbols()
    assert set(names) == {"sq_abi_version", "sq_status_str", "sq_quantize_int4_g128", "sq_quantize_fp8_e4m3",
                          "sq_qgemv_w4a16", "sq_qgemv_w8a16", "sq_verify_gemm_f16", "sq_spec_accept",
                          "sq_spec_accept_noalloc", "sq_probe_stream_read", "sq_embed_block_f16",
                          "sq_add_rmsnorm_f16", "sq_rope_kv_f16", "sq_attention_f16", "sq_silu_mul_f16",
                          "sq_spec_commit", "sq_spec_accept_multi", "sq_kv_adopt_f16", "sq_spec_commit_multi",
                          "sq_qgemv_w4a16_rmsnorm", "sq_verify_gemm_f16_rmsnorm", "sq_qgemv_w4a16_acc",
                          "sq_verify_gemm_f16_acc", "sq_qgemv_w4a16_rmsnorm_silu", "sq_rope_attention_f16"}
    assert set(names) == set(sq.EXPORTED)
    for n in names:
        assert hasattr(lib, n), n
    assert sq.sq_abi_version() == 7
    for s in range(9):
        assert lib.sq_status_str(s).startswith(b"SQ_")
    assert lib.sq_status_str(9) == b"unknown sq_status"


def test_quantize_validation():
    lib = sq.load()
    q4, q8 = lib.sq_quantize_int4_g128, lib.sq_quantize_fp8_e4m3
    assert q4(None, 4, 128, B, C, D, None, None) == NULL
    assert q4(A, 4, 100, B, C, D, None, None) == SHAPE
    assert q4(A, 0, 128, B, C, D, None, None) == SHAPE
    assert q4(A, 4, 1 << 21, B, C, D, None, None) == SHAPE
    assert q4(A + 2, 4, 128, B, C, D, None, None) == ALIGN
    assert q4(A, 4, 128, B + 8, C, D, None, None) == ALIGN
    assert q4(A, 4, 128, A + 16, C, D, None, None) == ALIAS       # codes inside w16
    assert q4(A, 4, 128, B, C, C + 2, None, None) == ALIAS        # zeros overlap scales
    assert q8(A, 4, 24, B, C, None, None) == SHAPE
    assert q8(A, 4, 32, B, C + 2, None, None) == ALIGN
    assert q8(A, 4, 32, B, A + 8, None, None) == ALIAS


def test_gemv_gemm_validation():
    lib = sq.load()
    w4, w8, gm = lib.sq_qgemv_w4a16, lib.sq_qgemv_w8a16, lib.sq_verify_gemm_f16
    assert w4(A, 1, 256, B, C, D, 10, None, F32, None) == NULL
    assert w4(A, 65, 256, B, C, D, 10, E, F32, None) == SHAPE
    assert w8(A, 65, 32, B, C, 10, E, F32, None) == SHAPE
    assert w4(A, 0, 256, B, C, D, 10, E, F32, None) == SHAPE
    assert w4(A, 1, 200, B, C, D, 10, E, F32, None) == SHAPE
    assert w4(A, 1, 256, B, C, D, 0, E, F32, None) == SHAPE
    assert w4(A, 1, 256, B, C, D, 10, E, 7, None) == UNSUPPORTED
    assert w4(A + 8, 1, 256, B, C, D, 10, E, F32, None) == ALIGN
    assert w4(A, 1, 256, B, C, D, 10, E + 2, F32, None) == ALIGN
    assert w4(A, 1, 256, B, C, D, 10, A + 64, F32, None) == ALIAS   # y overlaps x
    assert w8(A, 1, 24, B, C, 10, E, F32, None) == SHAPE
    assert w8(A, 1, 32, B, C + 2, 10, E, F32, None) == ALIGN
    assert w8(A, 2, 32, B, C, 10, C + 4, F16, None) == ALIAS        # y overlaps scales
    assert gm(A, 65, 64, B, 10, E, F32, None) == SHAPE
    assert gm(A, 5, 12, B, 10, E, F32, None) == SHAPE
    assert gm(A, 5, 64, B + 2, 10, E, F32, None) == ALIGN
    assert gm(A, 5, 64, B, 10, B + 100, F32, None) == ALIAS


def test_fused_projection_validation():
    """The decoder's fused projections validate on the host like the plain
    calls (plus the normalised source); a shape without a fused kernel is
    SQ_ERR_UNSUPPORTED, still without any HIP call."""
    lib = sq.load()
    n4, nf = lib.sq_qgemv_w4a16_rmsnorm, lib.sq_verify_gemm_f16_rmsnorm
    a4, af = lib.sq_qgemv_w4a16_acc, lib.sq_verify_gemm_f16_acc
    # (h, group, norm_w, eps, m, k, codes, scales, zeros, n, y, y_dtype, stream)
    assert n4(None, 1, A, 1e-6, 1, 256, B, C, D, 10, E, F32, None) == NULL
    assert n4(A, 1, None, 1e-6, 1, 256, B, C, D, 10, E, F32, None) == NULL
    assert n4(A, 0, C, 1e-6, 1, 256, B, C, D, 10, E, F32, None) == SHAPE
    assert n4(A, 1, C, float("nan"), 1, 256, B, C, D, 10, E, F32, None) == NONFINITE
    assert n4(A, 1, C, -1.0, 1, 256, B, C, D, 10, E, F32, None) == SHAPE
    assert n4(A, 1, C, 1e-6, 1, 32768, B, C, D, 10, E, F32, None) == SHAPE    # rows beyond 16384
    assert n4(A + 4, 1, C, 1e-6, 1, 256, B, C, D, 10, E, F32, None) == ALIGN
    assert n4(A, 1, C + 2, 1e-6, 1, 256, B, C + 1024, D, 10, E, F32, None) == ALIGN
    assert n4(A, 1, C, 1e-6, 1, 256, B, C + 1024, D, 10, A + 64, F32, None) == ALIAS   # y inside h
    assert n4(A, 1, C, 1e-6, 9, 256, B, C + 1024, D, 10, E, F32, None) == UNSUPPORTED  # m > 8
    # (h, group, norm_w, eps, m, k, w16, n, y, y_dtype, stream)
    assert nf(A, 1, C, 1e-6, 0, 64, B, 10, E, F32, None) == SHAPE
    assert nf(A, 1, C, 1e-6, 5, 64, B + 2, 10, E, F32, None) == ALIGN
    assert nf(A, 1, C, 1e-6, 5, 64, B, 10, B + 100, F32, None) == ALIAS
    assert nf(A, 1, C, 1e-6, 5, 64, B, 10, E, F32, None) == UNSUPPORTED  # 1280 bytes of weights: no row blocks
    # (x, m, k, codes, scales, zeros, n, y, stream) / (x, m, k, w16, n, y, stream)
    assert a4(A, 1, 256, B, C, D, 10, None, None) == NULL
    assert a4(A, 1, 256, B, C, D, 10, E + 2, None) == ALIGN
    assert a4(A, 1, 256, B, C, D, 10, A + 64, None) == ALIAS
    assert a4(A, 9, 256, B, C, D, 10, E, None) == UNSUPPORTED
    assert af(A, 5, 12, B, 10, E, None) == SHAPE
    assert af(A, 5, 64, B, 10, B + 100, None) == ALIAS
    assert af(A, 65, 64, B, 10, E, None) == SHAPE
    assert af(A, 5, 64, B, 10, E, None) == UNSUPPORTED


def test_accept_validation():
    lib = sq.load()
    acc = lib.sq_spec_accept
    # (draft, target, tokens, u24, b, kd, v, T, n_acc, next, q_out, p_out, stream)
    assert acc(A, None, C, D, 1, 4, 100, 1.0, E, E + 64, None, None, None) == NULL
    assert acc(None, B, C, D, 1, 4, 100, 1.0, E, E + 64, None, None, None) == NULL
    assert acc(A, B, C, None, 1, 4, 100, 1.0, E, E + 64, None, None, None) == NULL
    assert acc(A, B, C, D, 0, 4, 100, 1.0, E, E + 64, None, None, None) == SHAPE
    assert acc(A, B, C, D, 1, 65, 100, 1.0, E, E + 64, None, None, None) == SHAPE
    assert acc(A, B, C, D, 1, -1, 100, 1.0, E, E + 64, None, None, None) == SHAPE
    assert acc(A, B, C, D, 1, 4, 0, 1.0, E, E + 64, None, None, None) == SHAPE
    assert acc(A, B, C, D, 1 << 20, 8, 151936, 1.0, E, E + (1 << 22), None, None, None) == SHAPE
    assert acc(None, B, None, D, 1 << 24, 0, 1, 1.0, E, E + (1 << 26), None, None, None) == SHAPE
    assert acc(None, B, None, D, 1 << 23, 0, 4097, 1.0, E, E + (1 << 25), None, None, None) == SHAPE
    assert acc(A, B, C, D, 1, 1, (1 << 26) + 1, 1.0, E, E + 64, None, None, None) == SHAPE
    assert acc(A, B, C, D, 1, 4, 100, -1.0, E, E + 64, None, None, None) == UNSUPPORTED
    assert acc(A, B, C, D, 1, 4, 100, float("nan"), E, E + 64, None, None, None) == NONFINITE
    assert acc(A, B, C, D, 1, 4, 100, float("inf"), E, E + 64, None, None, None) == NONFINITE
    assert acc(A, B, C, D, 1, 4, 100, 0.0, E, E + 64, E + 128, None, None) == UNSUPPORTED
    assert acc(A, B, C, D, 1, 4, 100, 1.0, E + 2, E + 64, None, None, None) == ALIGN
    assert acc(A, B, C, D, 1, 4, 100, 1.0, E, E, None, None, None) == ALIAS
    assert acc(A, B, C, D, 1, 4, 100, 1.0, E, E + 64, None, B + 40, None) == ALIAS


def test_accept_noalloc_validation():
    """The allocation-free accept call validates like sq_spec_accept and
    rejects, on the host, calls whose scratch exceeds its static array."""
    lib = sq.load()
    acc, na = lib.sq_spec_accept, lib.sq_spec_accept_noalloc
    cases = [(A, None, C, D, 1, 4, 100, 1.0, E, E + 64, None, None, None),
             (A, B, C, D, 0, 4, 100, 1.0, E, E + 64, None, None, None),
             (A, B, C, D, 1, 4, 100, float("nan"), E, E + 64, None, None, None),
             (A, B, C, D, 1, 4, 100, 0.0, E, E + 64, E + 128, None, None),
             (A, B, C, D, 1, 4, 100, 1.0, E + 2, E + 64, None, None, None),
             (A, B, C, D, 1, 4, 100, 1.0, E, E, None, None, None)]
    for c in cases:
        assert na(*c) == acc(*c) != OK
    # 64 sequences at kd = 8 over 151936 logits need 2.7 MB: within the 4 MiB array (not launched here);
    # 100 need 4.3 MB: rejected before any HIP call
    assert na(A, B, C, D, 100, 8, 151936, 1.0, E, E + 4096, None, None, None) == SHAPE
    assert na(None, B, None, D, 300000, 0, 1, 1.0, E, E + (1 << 21), None, None, None) == SHAPE   # 16.8 MB


def test_probe_validation():
    probe = sq.load().sq_probe_stream_read
    assert probe(None, 1024, B, None) == NULL
    assert probe(A, 1024, None, None) == NULL
    assert probe(A, 0, B, None) == SHAPE
    assert probe(A, 1000, B, None) == SHAPE          # not a multiple of 16
    assert probe(A, (1 << 40) + 16, B, None) == SHAPE
    assert probe(A + 8, 1024, B, None) == ALIGN
    assert probe(A, 1024, B + 2, None) == ALIGN
    assert probe(A, 1024, A + 512, None) == ALIAS    # sink inside src
    assert probe(A + 8176, 1024, A, None) == ALIAS   # src starts inside the 8 KiB sink


def test_binding_fails_loudly_without_gpu_tensors():
    torch = pytest.importorskip("torch")
    with pytest.raises(ValueError):
        sq.sq_quantize_int4_g128(torch.zeros((4, 128), dtype=torch.float16))


def test_decoder_layer_validation():
    lib = sq.load()
    emb = lib.sq_embed_block_f16
    assert emb(None, 100, 64, B, None, 2, 0, C, None, None) == NULL
    assert emb(A, 100, 64, B, None, 2, 3, C, None, None) == NULL          # kd > 0 needs rest
    assert emb(A, 100, 60, B, None, 2, 0, C, None, None) == SHAPE         # hidden % 8
    assert emb(A, 100, 64, B, D, 2, 64, C, None, None) == SHAPE           # kd <= 63
    assert emb(A, 0, 64, B, None, 2, 0, C, None, None) == SHAPE
    assert emb(A + 8, 100, 64, B, None, 2, 0, C, None, None) == ALIGN
    assert emb(A, 100, 64, B, None, 2, 0, C + 4, None, None) == ALIGN
    assert emb(A, 100, 64, B, None, 2, 0, A + 256, None, None) == ALIAS    # h inside the table
    nrm = lib.sq_add_rmsnorm_f16
    assert nrm(A, None, 4, 64, None, 1e-6, 1, C, None) == NULL
    assert nrm(A, None, 5, 64, B, 1e-6, 2, C, None) == SHAPE              # m % group
    assert nrm(A, None, 4, 68, B, 1e-6, 1, C, None) == SHAPE
    assert nrm(A, None, 4, 64, B, float("nan"), 1, C, None) == NONFINITE
    assert nrm(A, None, 4, 64, B, -1.0, 1, C, None) == SHAPE
    assert nrm(A, D + 4, 4, 64, B, 1e-6, 1, C, None) == ALIGN
    assert nrm(A, None, 4, 64, B, 1e-6, 1, A + 512, None) == ALIAS        # x inside h
    assert nrm(A, A + 16, 4, 64, B, 1e-6, 1, C, None) == ALIAS            # delta overlaps h
    rope = lib.sq_rope_kv_f16
    args = dict(qkv=A, bias=None, b=1, rps=5, hq=28, hkv=4, pos=B, off=0, lb=1024, cap=1024, theta=1e6,
                q=C, kc=D, vc=E, st=None)

    def call(**kw):
        a = dict(args, **kw)
        return rope(a["qkv"], a["bias"], a["b"], a["rps"], a["hq"], a["hkv"], a["pos"], a["off"], a["lb"],
                    a["cap"], a["theta"], a["q"], a["kc"], a["vc"], a["st"], None)
    assert call(qkv=None) == NULL
    assert call(cap=1000, lb=1000) == SHAPE            # capacity % 64
    assert call(lb=2048) == SHAPE                      # len_bound > capacity
    assert call(hq=30) == SHAPE                        # hq % hkv
    assert call(rps=65) == SHAPE
    assert call(theta=float("inf")) == NONFINITE
    assert call(theta=1.0) == SHAPE
    assert call(pos=B + 2) == ALIGN
    assert call(q=D + 4096) == ALIAS                   # q_out inside the key cache
    assert call(vc=D + 64) == ALIAS                    # the two caches overlap
    ra = lib.sq_rope_attention_f16

    def fused(**kw):
        a = dict(args, **kw)
        return ra(a["qkv"], a["bias"], a["b"], a["rps"], a["hq"], a["hkv"], a["pos"], a["off"], a["lb"], a["cap"],
                  a["theta"], a["kc"], a["vc"], a["q"], a["st"], None)
    assert fused(q=None) == NULL                       # out
    assert fused(cap=1000, lb=1000) == SHAPE
    assert fused(theta=float("nan")) == NONFINITE
    assert fused(q=C + 2) == ALIGN
    assert fused(q=D + 4096) == ALIAS                  # out inside the key cache
    assert fused(qkv=E + 64) == ALIAS                  # the projection rows inside the value cache
    assert fused(rps=17, hq=8, hkv=8) == UNSUPPORTED   # more than 16 rows per sequence
    assert fused(rps=10) == UNSUPPORTED                # 70 query rows per kv head
    att = lib.sq_attention_f16
    assert att(A, None, E, 1, 5, 28, 4, B, 0, 1024, 1024, C, None) == NULL
    assert att(A, D, E, 1, 5, 28, 4, B, 0, 1024, 1000, C, None) == SHAPE
    assert att(A, D, E, 1, 5, 28, 4, B, 0, 0, 1024, C, None) == SHAPE
    assert att(A, D, E, 1, 5, 28, 4, B, 0, 1024, 1024, A + 128, None) == ALIAS   # out overlaps q
    assert att(A, D + 8, E, 1, 5, 28, 4, B, 0, 1024, 1024, C, None) == ALIGN
    silu = lib.sq_silu_mul_f16
    assert silu(None, 4, 8, B, None) == NULL
    assert silu(A, 1 << 21, 1 << 20, B, None) == SHAPE
    assert silu(A, 4, 8, A + 16, None) == ALIAS
    com = lib.sq_spec_commit
    assert com(A, B, None, 4, 3, C, D, E, None, 0, None, None, None) == NULL     # kd > 0 needs draft tokens
    assert com(A, B, A + 4096, 4, 3, C, D, E, C + 4096, 16, None, None, None) == NULL  # history needs out_len
    assert com(A, B, A + 4096, 0, 3, C, D, E, None, 0, None, None, None) == SHAPE
    assert com(A, B, A + 4096, 4, 65, C, D, E, None, 0, None, None, None) == SHAPE
    assert com(A, B, A + 4096, 4, 3, C, C + 8, E, None, 0, None, None, None) == ALIAS   # prev overlaps pending
    assert com(A, B, A + 4096, 4, 3, C, D, A + 4, None, 0, None, None, None) == ALIAS   # pos_base on n_accepted
    assert com(A, B, A + 4096, 4, 3, C + 2, D, E, None, 0, None, None, None) == ALIGN


def test_multi_chain_validation():
    lib = sq.load()
    acc = lib.sq_spec_accept_multi
    # draft, target, tokens, u24, b, c, kd, v, T, n, next, chain, q_out, p_out, stream
    assert acc(A, B, C, D, 2, 3, 4, 100, 1.0, E, E + 64, None, None, None, None) == NULL   # chain
    assert acc(A, B, C, D, 2, 65, 4, 100, 1.0, E, E + 64, E + 128, None, None, None) == SHAPE   # c <= 64
    assert acc(A, B, C, D, 2, 3, 65, 100, 1.0, E, E + 64, E + 128, None, None, None) == SHAPE   # kd <= 64
    assert acc(A, B, C, D, 2, 3, 4, 100, float("nan"), E, E + 64, E + 128, None, None, None) == NONFINITE
    assert acc(A, B, C, D, 2, 3, 4, 100, 0.0, E, E + 64, E + 128, E + 4096, None, None) == UNSUPPORTED
    assert acc(A, B, C, None, 2, 3, 4, 100, 1.0, E, E + 64, E + 128, None, None, None) == NULL   # u24 at T > 0
    assert acc(A, B, C, D, 2, 3, 4, 100, 1.0, E, E + 64, E + 130, None, None, None) == ALIGN
    assert acc(A, B, C, D, 2, 3, 4, 100, 1.0, E, E + 4, E + 128, None, None, None) == ALIAS    # next on n
    assert acc(A, B, C, D, 2, 3, 4, 100, 1.0, B + 64, E + 64, E + 128, None, None, None) == ALIAS  # n in target
    ad = lib.sq_kv_adopt_f16
    assert ad(None, B, 28, 1, 4, 4, 1024, C, D, E, 0, 0, None) == NULL
    assert ad(A, B, 28, 1, 65, 4, 1024, C, D, E, 0, 0, None) == SHAPE
    assert ad(A, B, 28, 1, 4, 4, 1000, C, D, E, 0, 0, None) == SHAPE
    assert ad(A, B, 28, 1, 4, 4, 1024, C, D, E, -65, 0, None) == SHAPE
    assert ad(A + 8, B, 28, 1, 4, 4, 1024, C, D, E, 0, 0, None) == ALIGN
    assert ad(A, A + 1024, 28, 1, 4, 4, 1024, C, D, E, 0, 0, None) == ALIAS   # the caches overlap
    cm = lib.sq_spec_commit_multi
    assert cm(A, B, C, None, 2, 3, 4, D, D + 4096, E, None, 0, None, None, None) == NULL     # drafts
    assert cm(A, B, C, A + 4096, 2, 0, 4, D, D + 4096, E, None, 0, None, None, None) == SHAPE
    assert cm(A, B, C, A + 4096, 2, 3, 4, D, D + 8, E, None, 0, None, None, None) == ALIAS   # prev on pending
    assert cm(A, B, C, A + 4096, 2, 3, 4, D + 2, D + 4096, E, None, 0, None, None, None) == ALIGN
