"""SpecQuant hot path on MI355X (gfx950): a C-ABI HIP library and its binding.

SpecQuant (arXiv 2609.21704) drafts tokens with quantized copies (INT4, FP8)
of one FP16 parent, verifies the drafted block with the parent and accepts or
corrects the drafted tokens.  The data-parallel steps of a round run in the
HIP kernels of ``libspecquant.so``; this package only marshals arguments
(``_lib``) and drives the calls of a round (``rounds`` for the
weight-streaming stack, ``decoder`` for the decoder with its cache).
"""
from ._lib import (  # noqa: F401
    EXPORTED,
    LIB_PATH,
    SQ_F16,
    SQ_F32,
    SpecQuantError,
    load,
    sq_abi_version,
    sq_add_rmsnorm_f16,
    sq_attention_f16,
    sq_embed_block_f16,
    sq_kv_adopt_f16,
    sq_qgemv_w4a16,
    sq_qgemv_w4a16_acc,
    sq_qgemv_w4a16_rmsnorm,
    sq_qgemv_w4a16_rmsnorm_silu,
    sq_qgemv_w8a16,
    sq_quantize_fp8_e4m3,
    sq_quantize_int4_g128,
    sq_probe_stream_read,
    sq_rope_attention_f16,
    sq_rope_kv_f16,
    sq_silu_mul_f16,
    sq_spec_accept,
    sq_spec_accept_multi,
    sq_spec_accept_noalloc,
    sq_spec_commit,
    sq_spec_commit_multi,
    sq_verify_gemm_f16,
    sq_verify_gemm_f16_acc,
    sq_verify_gemm_f16_rmsnorm,
)
