"""ctypes binding of libspecquant.so: argument marshalling only.

Each function has the name of the C entry point it calls (see
include/specquant.h).  Tensors supply device memory and the current torch
stream supplies the HIP stream; every computation runs in the library's HIP
kernels.  There is no fallback: if the library is not built, or a tensor is not
on the GPU, the call raises.
"""
from __future__ import annotations

import ctypes
import os
import threading

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libspecquant.so")

SQ_F16, SQ_F32 = 0, 1
_STATUS = {0: "SQ_OK", 1: "SQ_ERR_NULL", 2: "SQ_ERR_SHAPE", 3: "SQ_ERR_ALIGN", 4: "SQ_ERR_ALIAS",
           5: "SQ_ERR_NONFINITE", 6: "SQ_ERR_UNSUPPORTED", 7: "SQ_ERR_DEVICE", 8: "SQ_ERR_CAPTURE"}

_lib = None
_lock = threading.Lock()


class SpecQuantError(RuntimeError):
    def __init__(self, status: int, fn: str):
        self.status = status
        super().__init__(f"{fn} failed: {_STATUS.get(status, status)}")


def load() -> ctypes.CDLL:
    """Load the built library (raises if it has not been built)."""
    global _lib
    with _lock:
        if _lib is not None:
            return _lib
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                               "(the SpecQuant path has no non-HIP fallback)")
        lib = ctypes.CDLL(LIB_PATH)
        P, I64, I32, F = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_float
        S = ctypes.c_int
        sigs = {
            "sq_abi_version": ([], I32),
            "sq_status_str": ([S], ctypes.c_char_p),
            "sq_quantize_int4_g128": ([P, I64, I64, P, P, P, P, P], S),
            "sq_quantize_fp8_e4m3": ([P, I64, I64, P, P, P, P], S),
            "sq_qgemv_w4a16": ([P, I64, I64, P, P, P, I64, P, S, P], S),
            "sq_qgemv_w8a16": ([P, I64, I64, P, P, I64, P, S, P], S),
            "sq_verify_gemm_f16": ([P, I64, I64, P, I64, P, S, P], S),
            "sq_spec_accept": ([P, P, P, P, I32, I32, I32, F, P, P, P, P, P], S),
            "sq_spec_accept_noalloc": ([P, P, P, P, I32, I32, I32, F, P, P, P, P, P], S),
            "sq_probe_stream_read": ([P, I64, P, P], S),
            "sq_embed_block_f16": ([P, I64, I64, P, P, I32, I32, P, P, P], S),
            "sq_add_rmsnorm_f16": ([P, P, I64, I64, P, F, I32, P, P], S),
            "sq_rope_kv_f16": ([P, P, I32, I32, I32, I32, P, I32, I64, I64, ctypes.c_double, P, P, P, P, P], S),
            "sq_attention_f16": ([P, P, P, I32, I32, I32, I32, P, I32, I64, I64, P, P], S),
            "sq_rope_attention_f16": ([P, P, I32, I32, I32, I32, P, I32, I64, I64, ctypes.c_double, P, P, P, P, P],
                                      S),
            "sq_silu_mul_f16": ([P, I64, I64, P, P], S),
            "sq_qgemv_w4a16_rmsnorm": ([P, I32, P, F, I64, I64, P, P, P, I64, P, S, P], S),
            "sq_verify_gemm_f16_rmsnorm": ([P, I32, P, F, I64, I64, P, I64, P, S, P], S),
            "sq_qgemv_w4a16_acc": ([P, I64, I64, P, P, P, I64, P, P], S),
            "sq_qgemv_w4a16_rmsnorm_silu": ([P, I32, P, F, I64, I64, P, P, P, I64, P, P], S),
            "sq_verify_gemm_f16_acc": ([P, I64, I64, P, I64, P, P], S),
            "sq_spec_commit": ([P, P, P, I32, I32, P, P, P, P, I64, P, P, P], S),
            "sq_spec_accept_multi": ([P, P, P, P, I32, I32, I32, I32, F, P, P, P, P, P, P], S),
            "sq_kv_adopt_f16": ([P, P, I32, I32, I32, I32, I64, P, P, P, I32, I32, P], S),
            "sq_spec_commit_multi": ([P, P, P, P, I32, I32, I32, P, P, P, P, I64, P, P, P], S),
        }
        for name, (args, res) in sigs.items():
            fn = getattr(lib, name)
            fn.argtypes = args
            fn.restype = res
        _lib = lib
        return lib


EXPORTED = ("sq_abi_version", "sq_status_str", "sq_quantize_int4_g128", "sq_quantize_fp8_e4m3",
            "sq_qgemv_w4a16", "sq_qgemv_w8a16", "sq_verify_gemm_f16", "sq_spec_accept",
            "sq_spec_accept_noalloc", "sq_probe_stream_read", "sq_embed_block_f16", "sq_add_rmsnorm_f16",
            "sq_rope_kv_f16", "sq_attention_f16", "sq_silu_mul_f16", "sq_spec_commit", "sq_spec_accept_multi",
            "sq_kv_adopt_f16", "sq_spec_commit_multi", "sq_qgemv_w4a16_rmsnorm", "sq_verify_gemm_f16_rmsnorm",
            "sq_qgemv_w4a16_acc", "sq_verify_gemm_f16_acc", "sq_qgemv_w4a16_rmsnorm_silu",
            "sq_rope_attention_f16")

# device status bits (SQ_DEV_* of include/specquant.h)
DEV_BAD_TOKEN, DEV_BAD_POS, DEV_OVERFLOW, DEV_NO_DIST = 1, 2, 4, 8


def _ptr(t):
    return None if t is None else t.data_ptr()


def _stream(dev: torch.device):
    return torch.cuda.current_stream(dev).cuda_stream


def _dev(*ts):
    dev = None
    for t in ts:
        if t is None:
            continue
        if not t.is_cuda:
            raise ValueError("SpecQuant calls take GPU tensors only")
        if not t.is_contiguous():
            raise ValueError("SpecQuant calls take contiguous tensors only")
        if dev is None:
            dev = t.device
        elif t.device != dev:
            raise ValueError("all tensors of a call must be on one device")
    return dev


def _check(status: int, fn: str):
    if status != 0:
        raise SpecQuantError(status, fn)


def _dtype_code(dt: torch.dtype) -> int:
    if dt == torch.float16:
        return SQ_F16
    if dt == torch.float32:
        return SQ_F32
    raise ValueError("output dtype must be torch.float16 or torch.float32")


def _expect(t, dtype, shape, name):
    if t.dtype != dtype:
        raise TypeError(f"{name}: expected {dtype}, got {t.dtype}")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name}: expected shape {tuple(shape)}, got {tuple(t.shape)}")


def sq_abi_version() -> int:
    return int(load().sq_abi_version())


def sq_quantize_int4_g128(w16: torch.Tensor, codes=None, scales=None, zeros=None, nonfinite_flag=None):
    """FP16 parent [n][k] -> (codes u8 [n][k/2], scales f16 [n][k/128], zeros f16 [n][k/128])."""
    n, k = w16.shape
    if w16.dtype != torch.float16:
        raise TypeError("w16 must be float16")
    dev = w16.device
    codes = torch.empty((n, k // 2), dtype=torch.uint8, device=dev) if codes is None else codes
    scales = torch.empty((n, k // 128), dtype=torch.float16, device=dev) if scales is None else scales
    zeros = torch.empty((n, k // 128), dtype=torch.float16, device=dev) if zeros is None else zeros
    _dev(w16, codes, scales, zeros, nonfinite_flag)
    _expect(codes, torch.uint8, (n, k // 2), "codes")
    _expect(scales, torch.float16, (n, k // 128), "scales")
    _expect(zeros, torch.float16, (n, k // 128), "zeros")
    _check(load().sq_quantize_int4_g128(_ptr(w16), n, k, _ptr(codes), _ptr(scales), _ptr(zeros),
                                        _ptr(nonfinite_flag), _stream(dev)), "sq_quantize_int4_g128")
    return codes, scales, zeros


def sq_quantize_fp8_e4m3(w16: torch.Tensor, codes=None, scales=None, nonfinite_flag=None):
    """FP16 parent [n][k] -> (codes u8 [n][k] OCP E4M3, scales f32 [n])."""
    n, k = w16.shape
    if w16.dtype != torch.float16:
        raise TypeError("w16 must be float16")
    dev = w16.device
    codes = torch.empty((n, k), dtype=torch.uint8, device=dev) if codes is None else codes
    scales = torch.empty((n,), dtype=torch.float32, device=dev) if scales is None else scales
    _dev(w16, codes, scales, nonfinite_flag)
    _expect(codes, torch.uint8, (n, k), "codes")
    _expect(scales, torch.float32, (n,), "scales")
    _check(load().sq_quantize_fp8_e4m3(_ptr(w16), n, k, _ptr(codes), _ptr(scales), _ptr(nonfinite_flag),
                                       _stream(dev)), "sq_quantize_fp8_e4m3")
    return codes, scales


def sq_qgemv_w4a16(x, codes, scales, zeros, y=None, y_dtype=torch.float32):
    """y[m][n] = x . W4'^T with W4' the INT4 g128 dequantized weights."""
    m, k = x.shape
    n = codes.shape[0]
    if x.dtype != torch.float16:
        raise TypeError("x must be float16")
    y = torch.empty((m, n), dtype=y_dtype, device=x.device) if y is None else y
    _dev(x, codes, scales, zeros, y)
    _expect(codes, torch.uint8, (n, k // 2), "codes")
    _expect(scales, torch.float16, (n, k // 128), "scales")
    _expect(zeros, torch.float16, (n, k // 128), "zeros")
    if y.numel() != m * n:
        raise ValueError("y must hold m * n elements")
    _check(load().sq_qgemv_w4a16(_ptr(x), m, k, _ptr(codes), _ptr(scales), _ptr(zeros), n, _ptr(y),
                                 _dtype_code(y.dtype), _stream(x.device)), "sq_qgemv_w4a16")
    return y


SQ_ERR_UNSUPPORTED = 6


def _fused(status: int, fn: str) -> bool:
    """True when the fused call ran; False when its shape has no fused form (nothing enqueued)."""
    if status == SQ_ERR_UNSUPPORTED:
        return False
    _check(status, fn)
    return True


def _norm_src(h, norm_w, group: int):
    if h.dtype != torch.float32 or h.dim() != 2 or h.shape[0] % group:
        raise ValueError("h must be float32 [m * group][k]")
    _expect(norm_w, torch.float16, (h.shape[1],), "norm_w")
    return h.shape[0] // group, h.shape[1]


def sq_qgemv_w4a16_rmsnorm(h, norm_w, eps: float, codes, scales, zeros, group: int = 1, y=None,
                           y_dtype=torch.float32) -> bool:
    """y = x . W4'^T with x the rows sq_add_rmsnorm_f16(h, norm_w, eps, group) writes, normalised inside the
    projection; False (nothing enqueued) where the projection's kernel has no such form."""
    m, k = _norm_src(h, norm_w, group)
    n = codes.shape[0]
    _dev(h, norm_w, codes, scales, zeros, y)
    _expect(codes, torch.uint8, (n, k // 2), "codes")
    _expect(scales, torch.float16, (n, k // 128), "scales")
    _expect(zeros, torch.float16, (n, k // 128), "zeros")
    if y.numel() != m * n:
        raise ValueError("y must hold m * n elements")
    return _fused(load().sq_qgemv_w4a16_rmsnorm(_ptr(h), int(group), _ptr(norm_w), float(eps), m, k, _ptr(codes),
                                                _ptr(scales), _ptr(zeros), n, _ptr(y), _dtype_code(y.dtype),
                                                _stream(h.device)), "sq_qgemv_w4a16_rmsnorm")


def sq_qgemv_w4a16_rmsnorm_silu(h, norm_w, eps: float, codes, scales, zeros, t, group: int = 1) -> bool:
    """t = f16(silu(g) * u) with g | u = x . W4'^T the gate and up halves of the fused gate|up rows and x the
    rows sq_add_rmsnorm_f16(h, norm_w, eps, group) writes; False (nothing enqueued) where the projection's
    kernel has no such form."""
    m, k = _norm_src(h, norm_w, group)
    n = codes.shape[0]
    _dev(h, norm_w, codes, scales, zeros, t)
    _expect(codes, torch.uint8, (n, k // 2), "codes")
    _expect(scales, torch.float16, (n, k // 128), "scales")
    _expect(zeros, torch.float16, (n, k // 128), "zeros")
    if t.dtype != torch.float16 or t.numel() != m * (n // 2):
        raise ValueError("t must be float16 with m * n / 2 elements")
    return _fused(load().sq_qgemv_w4a16_rmsnorm_silu(_ptr(h), int(group), _ptr(norm_w), float(eps), m, k,
                                                     _ptr(codes), _ptr(scales), _ptr(zeros), n, _ptr(t),
                                                     _stream(h.device)), "sq_qgemv_w4a16_rmsnorm_silu")


def sq_verify_gemm_f16_rmsnorm(h, norm_w, eps: float, w16, group: int = 1, y=None) -> bool:
    """y = x . W16^T with x the rows sq_add_rmsnorm_f16(h, norm_w, eps, group) writes, normalised inside the
    projection; False (nothing enqueued) where the projection's kernel has no such form."""
    m, k = _norm_src(h, norm_w, group)
    n = w16.shape[0]
    _dev(h, norm_w, w16, y)
    _expect(w16, torch.float16, (n, k), "w16")
    if y.numel() != m * n:
        raise ValueError("y must hold m * n elements")
    return _fused(load().sq_verify_gemm_f16_rmsnorm(_ptr(h), int(group), _ptr(norm_w), float(eps), m, k, _ptr(w16),
                                                    n, _ptr(y), _dtype_code(y.dtype), _stream(h.device)),
                  "sq_verify_gemm_f16_rmsnorm")


def sq_qgemv_w4a16_acc(x, codes, scales, zeros, y) -> bool:
    """y += x . W4'^T (y float32); False (nothing enqueued) where the projection's kernel has no such form."""
    m, k = x.shape
    n = codes.shape[0]
    if x.dtype != torch.float16 or y.dtype != torch.float32 or y.numel() != m * n:
        raise ValueError("x must be float16 [m][k] and y float32 with m * n elements")
    _dev(x, codes, scales, zeros, y)
    _expect(codes, torch.uint8, (n, k // 2), "codes")
    _expect(scales, torch.float16, (n, k // 128), "scales")
    _expect(zeros, torch.float16, (n, k // 128), "zeros")
    return _fused(load().sq_qgemv_w4a16_acc(_ptr(x), m, k, _ptr(codes), _ptr(scales), _ptr(zeros), n, _ptr(y),
                                            _stream(x.device)), "sq_qgemv_w4a16_acc")


def sq_verify_gemm_f16_acc(x, w16, y) -> bool:
    """y += x . W16^T (y float32); False (nothing enqueued) where the projection's kernel has no such form."""
    m, k = x.shape
    n = w16.shape[0]
    if x.dtype != torch.float16 or y.dtype != torch.float32 or y.numel() != m * n:
        raise ValueError("x must be float16 [m][k] and y float32 with m * n elements")
    _dev(x, w16, y)
    _expect(w16, torch.float16, (n, k), "w16")
    return _fused(load().sq_verify_gemm_f16_acc(_ptr(x), m, k, _ptr(w16), n, _ptr(y), _stream(x.device)),
                  "sq_verify_gemm_f16_acc")


def sq_qgemv_w8a16(x, codes, scales, y=None, y_dtype=torch.float32):
    """y[m][n] = x . W8'^T with W8' the FP8 E4M3 dequantized weights."""
    m, k = x.shape
    n = codes.shape[0]
    if x.dtype != torch.float16:
        raise TypeError("x must be float16")
    y = torch.empty((m, n), dtype=y_dtype, device=x.device) if y is None else y
    _dev(x, codes, scales, y)
    _expect(codes, torch.uint8, (n, k), "codes")
    _expect(scales, torch.float32, (n,), "scales")
    if y.numel() != m * n:
        raise ValueError("y must hold m * n elements")
    _check(load().sq_qgemv_w8a16(_ptr(x), m, k, _ptr(codes), _ptr(scales), n, _ptr(y), _dtype_code(y.dtype),
                                 _stream(x.device)), "sq_qgemv_w8a16")
    return y


def sq_verify_gemm_f16(x, w16, y=None, y_dtype=torch.float32):
    """y[m][n] = x . W16^T (parent verification pass)."""
    m, k = x.shape
    n = w16.shape[0]
    if x.dtype != torch.float16 or w16.dtype != torch.float16:
        raise TypeError("x and w16 must be float16")
    y = torch.empty((m, n), dtype=y_dtype, device=x.device) if y is None else y
    _dev(x, w16, y)
    _expect(w16, torch.float16, (n, k), "w16")
    if y.numel() != m * n:
        raise ValueError("y must hold m * n elements")
    _check(load().sq_verify_gemm_f16(_ptr(x), m, k, _ptr(w16), n, _ptr(y), _dtype_code(y.dtype),
                                     _stream(x.device)), "sq_verify_gemm_f16")
    return y


def sq_spec_accept(draft_logits, target_logits, draft_tokens, u24, temperature: float = 1.0,
                   n_accepted=None, next_token=None, q_out=None, p_out=None, _entry="sq_spec_accept"):
    """Speculative accept / resample.

    draft_logits [kd][b][v] f32 (None when kd == 0), target_logits [b][kd+1][v] f32,
    draft_tokens [kd][b] int32, u24 [b][kd+1] int32 holding uint32 bit patterns
    (low 24 bits used).  Returns (n_accepted [b] int32, next_token [b] int32).
    """
    b, kd1, v = target_logits.shape
    kd = kd1 - 1
    dev = target_logits.device
    n_accepted = torch.empty((b,), dtype=torch.int32, device=dev) if n_accepted is None else n_accepted
    next_token = torch.empty((b,), dtype=torch.int32, device=dev) if next_token is None else next_token
    _dev(draft_logits, target_logits, draft_tokens, u24, n_accepted, next_token, q_out, p_out)
    if target_logits.dtype != torch.float32 or (draft_logits is not None and draft_logits.dtype != torch.float32):
        raise TypeError("logits must be float32")
    if draft_logits is not None and draft_logits.numel() != kd * b * v:
        raise ValueError("draft_logits must be [kd][b][v]")
    if draft_tokens is not None and (draft_tokens.dtype != torch.int32 or draft_tokens.numel() != b * kd):
        raise ValueError("draft_tokens must be int32 [kd][b]")
    if u24 is not None and (u24.dtype != torch.int32 or u24.numel() != b * (kd + 1)):
        raise ValueError("u24 must be int32 [b][kd+1]")
    _expect(n_accepted, torch.int32, (b,), "n_accepted")
    _expect(next_token, torch.int32, (b,), "next_token")
    if q_out is not None:
        _expect(q_out, torch.float32, (kd, b, v), "q_out")
    if p_out is not None:
        _expect(p_out, torch.float32, (b, kd + 1, v), "p_out")
    fn = getattr(load(), _entry)
    _check(fn(_ptr(draft_logits), _ptr(target_logits), _ptr(draft_tokens), _ptr(u24), b, kd, v, float(temperature),
              _ptr(n_accepted), _ptr(next_token), _ptr(q_out), _ptr(p_out), _stream(dev)), _entry)
    return n_accepted, next_token


NOALLOC_SCRATCH_BYTES = 4 << 20  # SQ_NOALLOC_SCRATCH_BYTES


def sq_spec_accept_noalloc(draft_logits, target_logits, draft_tokens, u24, temperature: float = 1.0,
                           n_accepted=None, next_token=None, q_out=None, p_out=None):
    """sq_spec_accept without any device allocation by the library (its
    scratch is a static per-GPU array of NOALLOC_SCRATCH_BYTES); same
    arguments and results.  Pass n_accepted / next_token (and any q_out /
    p_out) to keep the call itself free of torch allocations too."""
    return sq_spec_accept(draft_logits, target_logits, draft_tokens, u24, temperature, n_accepted, next_token,
                          q_out, p_out, _entry="sq_spec_accept_noalloc")


PROBE_SINK_WORDS = 2048  # SQ_PROBE_SINK_WORDS


def sq_probe_stream_read(src: torch.Tensor, nbytes: int | None = None, offset: int = 0, sink=None):
    """Streaming-read probe (a measurement aid, not a step of the method): one
    plain read of `nbytes` bytes of the GPU tensor `src` from byte `offset` on
    (default: all of it).  Returns the sink, uint32 words held in an int32
    tensor [PROBE_SINK_WORDS] whose XOR is the XOR of the 32-bit words read."""
    dev = src.device
    total = src.numel() * src.element_size()
    nbytes = total - offset if nbytes is None else nbytes
    if offset < 0 or nbytes < 0 or offset + nbytes > total:
        raise ValueError("byte range outside src")
    sink = torch.empty((PROBE_SINK_WORDS,), dtype=torch.int32, device=dev) if sink is None else sink
    _dev(src, sink)
    _expect(sink, torch.int32, (PROBE_SINK_WORDS,), "sink")
    _check(load().sq_probe_stream_read(src.data_ptr() + offset, nbytes, sink.data_ptr(), _stream(dev)),
           "sq_probe_stream_read")
    return sink


# ------------------------------------------------------------ decoder layer
HEAD_DIM = 128


def sq_embed_block_f16(table, first, rest=None, h=None, status=None):
    """h [b][kd+1][hidden] f32 = table[tokens] for the block (first [b], rest [kd][b])."""
    vocab, hidden = table.shape
    b = first.shape[0]
    kd = 0 if rest is None else rest.shape[0]
    h = torch.empty((b, kd + 1, hidden), dtype=torch.float32, device=table.device) if h is None else h
    _dev(table, first, rest, h, status)
    _expect(table, torch.float16, (vocab, hidden), "table")
    _expect(first, torch.int32, (b,), "first")
    if rest is not None:
        _expect(rest, torch.int32, (kd, b), "rest")
    if h.dtype != torch.float32 or h.numel() != b * (kd + 1) * hidden:
        raise ValueError("h must be float32 [b][kd+1][hidden]")
    _check(load().sq_embed_block_f16(_ptr(table), vocab, hidden, _ptr(first), _ptr(rest), b, kd, _ptr(h),
                                     _ptr(status), _stream(table.device)), "sq_embed_block_f16")
    return h


def sq_add_rmsnorm_f16(h, w, eps: float, delta=None, group: int = 1, x=None):
    """h += delta (in place); x = f16(rmsnorm(h rows group-1, 2 group-1, ...))."""
    hidden = w.shape[0]
    m = h.numel() // hidden
    x = torch.empty((m // group, hidden), dtype=torch.float16, device=h.device) if x is None else x
    _dev(h, w, delta, x)
    if h.dtype != torch.float32 or h.numel() != m * hidden:
        raise ValueError("h must be float32 [m][hidden]")
    if delta is not None and (delta.dtype != torch.float32 or delta.numel() != m * hidden):
        raise ValueError("delta must be float32 [m][hidden]")
    _expect(w, torch.float16, (hidden,), "w")
    if x.dtype != torch.float16 or x.numel() != (m // group) * hidden:
        raise ValueError("x must be float16 [m / group][hidden]")
    _check(load().sq_add_rmsnorm_f16(_ptr(h), _ptr(delta), m, hidden, _ptr(w), float(eps), int(group), _ptr(x),
                                     _stream(h.device)), "sq_add_rmsnorm_f16")
    return x


def _cache_dims(k_cache, v_cache):
    b, hkv, cap, hd = k_cache.shape
    if hd != HEAD_DIM:
        raise ValueError("k_cache must be [b][hkv][capacity][128]")
    _expect(v_cache, torch.float16, (b, hkv, HEAD_DIM, cap), "v_cache")
    if k_cache.dtype != torch.float16:
        raise TypeError("k_cache must be float16")
    return b, hkv, cap


def sq_rope_kv_f16(qkv, bias, pos_base, pos_offset: int, rows_per_seq: int, hq: int, k_cache, v_cache,
                   len_bound: int | None = None, theta: float = 1e6, q_out=None, status=None):
    """Bias + RoPE of the q|k|v rows, keys and values into the cache; returns q_out [m][hq][128] fp16."""
    b, hkv, cap = _cache_dims(k_cache, v_cache)
    m = b * rows_per_seq
    nh = hq + 2 * hkv
    len_bound = cap if len_bound is None else len_bound
    q_out = torch.empty((m, hq, HEAD_DIM), dtype=torch.float16, device=qkv.device) if q_out is None else q_out
    _dev(qkv, bias, pos_base, q_out, k_cache, v_cache, status)
    if qkv.dtype != torch.float32 or qkv.numel() != m * nh * HEAD_DIM:
        raise ValueError("qkv must be float32 [m][(hq + 2 hkv) * 128]")
    if bias is not None:
        _expect(bias, torch.float16, (nh * HEAD_DIM,), "bias")
    _expect(pos_base, torch.int32, (b,), "pos_base")
    _expect(q_out, torch.float16, (m, hq, HEAD_DIM), "q_out")
    _check(load().sq_rope_kv_f16(_ptr(qkv), _ptr(bias), b, rows_per_seq, hq, hkv, _ptr(pos_base), int(pos_offset),
                                 int(len_bound), cap, float(theta), _ptr(q_out), _ptr(k_cache), _ptr(v_cache),
                                 _ptr(status), _stream(qkv.device)), "sq_rope_kv_f16")
    return q_out


def sq_attention_f16(q, k_cache, v_cache, pos_base, pos_offset: int, rows_per_seq: int,
                     len_bound: int | None = None, out=None):
    """Causal GQA attention of the block rows over the cache; returns out [m][hq][128] fp16."""
    b, hkv, cap = _cache_dims(k_cache, v_cache)
    m, hq, hd = q.shape
    if hd != HEAD_DIM or m != b * rows_per_seq:
        raise ValueError("q must be [b * rows_per_seq][hq][128]")
    len_bound = cap if len_bound is None else len_bound
    out = torch.empty((m, hq, HEAD_DIM), dtype=torch.float16, device=q.device) if out is None else out
    _dev(q, k_cache, v_cache, pos_base, out)
    if q.dtype != torch.float16:
        raise TypeError("q must be float16")
    _expect(pos_base, torch.int32, (b,), "pos_base")
    if out.dtype != torch.float16 or out.numel() != m * hq * HEAD_DIM:
        raise ValueError("out must be float16 [m][hq][128]")
    _check(load().sq_attention_f16(_ptr(q), _ptr(k_cache), _ptr(v_cache), b, rows_per_seq, hq, hkv, _ptr(pos_base),
                                   int(pos_offset), int(len_bound), cap, _ptr(out), _stream(q.device)),
           "sq_attention_f16")
    return out


def sq_rope_attention_f16(qkv, bias, pos_base, pos_offset: int, rows_per_seq: int, hq: int, k_cache, v_cache,
                          out, len_bound: int | None = None, theta: float = 1e6, status=None) -> bool:
    """sq_rope_kv_f16 then sq_attention_f16 in one call (no q_out), the same bits; False (nothing enqueued)
    for blocks the fused kernel does not take."""
    b, hkv, cap = _cache_dims(k_cache, v_cache)
    m = b * rows_per_seq
    nh = hq + 2 * hkv
    len_bound = cap if len_bound is None else len_bound
    _dev(qkv, bias, pos_base, k_cache, v_cache, out, status)
    if qkv.dtype != torch.float32 or qkv.numel() != m * nh * HEAD_DIM:
        raise ValueError("qkv must be float32 [m][(hq + 2 hkv) * 128]")
    if bias is not None:
        _expect(bias, torch.float16, (nh * HEAD_DIM,), "bias")
    _expect(pos_base, torch.int32, (b,), "pos_base")
    if out.dtype != torch.float16 or out.numel() != m * hq * HEAD_DIM:
        raise ValueError("out must be float16 [m][hq][128]")
    return _fused(load().sq_rope_attention_f16(_ptr(qkv), _ptr(bias), b, rows_per_seq, hq, hkv, _ptr(pos_base),
                                               int(pos_offset), int(len_bound), cap, float(theta), _ptr(k_cache),
                                               _ptr(v_cache), _ptr(out), _ptr(status), _stream(qkv.device)),
                  "sq_rope_attention_f16")


def sq_silu_mul_f16(gu, t=None):
    """t [m][I] fp16 = silu(gate) * up of gu [m][2 I] f32."""
    m, two_i = gu.shape
    inter = two_i // 2
    t = torch.empty((m, inter), dtype=torch.float16, device=gu.device) if t is None else t
    _dev(gu, t)
    if gu.dtype != torch.float32 or two_i % 2:
        raise ValueError("gu must be float32 [m][2 I]")
    if t.dtype != torch.float16 or t.numel() != m * inter:
        raise ValueError("t must be float16 [m][I]")
    _check(load().sq_silu_mul_f16(_ptr(gu), m, inter, _ptr(t), _stream(gu.device)), "sq_silu_mul_f16")
    return t


def sq_spec_commit(n_accepted, next_token, draft_tokens, pending, prev, pos_base, out_tokens=None, out_len=None,
                   status=None):
    """Commit a round: append the emitted tokens, move pending / prev / pos_base."""
    b = n_accepted.shape[0]
    kd = 0 if draft_tokens is None else draft_tokens.shape[0]
    _dev(n_accepted, next_token, draft_tokens, pending, prev, pos_base, out_tokens, out_len, status)
    for t, name in ((n_accepted, "n_accepted"), (next_token, "next_token"), (pending, "pending"), (prev, "prev"),
                    (pos_base, "pos_base")):
        _expect(t, torch.int32, (b,), name)
    if draft_tokens is not None:
        _expect(draft_tokens, torch.int32, (kd, b), "draft_tokens")
    cap = 0
    if out_tokens is not None:
        if out_tokens.dtype != torch.int32 or out_tokens.dim() != 2 or out_tokens.shape[0] != b:
            raise ValueError("out_tokens must be int32 [b][capacity]")
        cap = out_tokens.shape[1]
        _expect(out_len, torch.int32, (b,), "out_len")
    _check(load().sq_spec_commit(_ptr(n_accepted), _ptr(next_token), _ptr(draft_tokens), b, kd, _ptr(pending),
                                 _ptr(prev), _ptr(pos_base), _ptr(out_tokens), cap, _ptr(out_len), _ptr(status),
                                 _stream(n_accepted.device)), "sq_spec_commit")


# ------------------------------------------------------ several draft chains
def sq_spec_accept_multi(draft_logits, target_logits, draft_tokens, u24, temperature: float = 1.0,
                         n_accepted=None, next_token=None, chain=None, q_out=None, p_out=None):
    """Multi-candidate accept / correct: draft_logits [kd][b][c][v],
    target_logits [b][c][kd+1][v] f32, draft_tokens [kd][b][c] int32,
    u24 [b][c kd + 1] int32 (uint32 bits).  Returns (n_accepted, next_token, chain)."""
    b, c, kd1, v = target_logits.shape
    kd = kd1 - 1
    dev = target_logits.device
    n_accepted = torch.empty((b,), dtype=torch.int32, device=dev) if n_accepted is None else n_accepted
    next_token = torch.empty((b,), dtype=torch.int32, device=dev) if next_token is None else next_token
    chain = torch.empty((b,), dtype=torch.int32, device=dev) if chain is None else chain
    _dev(draft_logits, target_logits, draft_tokens, u24, n_accepted, next_token, chain, q_out, p_out)
    if target_logits.dtype != torch.float32 or (draft_logits is not None and draft_logits.dtype != torch.float32):
        raise TypeError("logits must be float32")
    if draft_logits is not None and draft_logits.numel() != kd * b * c * v:
        raise ValueError("draft_logits must be [kd][b][c][v]")
    if draft_tokens is not None and (draft_tokens.dtype != torch.int32 or draft_tokens.numel() != kd * b * c):
        raise ValueError("draft_tokens must be int32 [kd][b][c]")
    if u24 is not None and (u24.dtype != torch.int32 or u24.numel() != b * (c * kd + 1)):
        raise ValueError("u24 must be int32 [b][c kd + 1]")
    for t, name in ((n_accepted, "n_accepted"), (next_token, "next_token"), (chain, "chain")):
        _expect(t, torch.int32, (b,), name)
    if q_out is not None:
        _expect(q_out, torch.float32, (kd, b, c, v), "q_out")
    if p_out is not None:
        _expect(p_out, torch.float32, (b, c, kd + 1, v), "p_out")
    _check(load().sq_spec_accept_multi(_ptr(draft_logits), _ptr(target_logits), _ptr(draft_tokens), _ptr(u24), b, c,
                                       kd, v, float(temperature), _ptr(n_accepted), _ptr(next_token), _ptr(chain),
                                       _ptr(q_out), _ptr(p_out), _stream(dev)), "sq_spec_accept_multi")
    return n_accepted, next_token, chain


def sq_kv_adopt_f16(k_cache, v_cache, b: int, c: int, chain, n_accepted, pos_base, lo_offset: int, hi_offset: int):
    """Copy the accepted chain's cache entries to the other chains:
    k_cache [layers][b c][hkv][capacity][128], v_cache [layers][b c][hkv][128][capacity]."""
    layers, bc, hkv, cap, hd = k_cache.shape
    if bc != b * c or hd != HEAD_DIM:
        raise ValueError("k_cache must be [layers][b c][hkv][capacity][128]")
    _expect(v_cache, torch.float16, (layers, bc, hkv, HEAD_DIM, cap), "v_cache")
    _dev(k_cache, v_cache, chain, n_accepted, pos_base)
    _expect(chain, torch.int32, (b,), "chain")
    _expect(n_accepted, torch.int32, (b,), "n_accepted")
    _expect(pos_base, torch.int32, (bc,), "pos_base")
    _check(load().sq_kv_adopt_f16(_ptr(k_cache), _ptr(v_cache), layers, b, c, hkv, cap, _ptr(chain), _ptr(n_accepted),
                                  _ptr(pos_base), int(lo_offset), int(hi_offset), _stream(k_cache.device)),
           "sq_kv_adopt_f16")


def sq_spec_commit_multi(n_accepted, next_token, chain, draft_tokens, c: int, pending, prev, pos_base,
                         out_tokens=None, out_len=None, status=None):
    """Commit a round of c chains per sequence (pending / prev / pos_base are [b c])."""
    b = n_accepted.shape[0]
    kd = 0 if draft_tokens is None else draft_tokens.shape[0]
    _dev(n_accepted, next_token, chain, draft_tokens, pending, prev, pos_base, out_tokens, out_len, status)
    for t, name in ((n_accepted, "n_accepted"), (next_token, "next_token"), (chain, "chain")):
        _expect(t, torch.int32, (b,), name)
    for t, name in ((pending, "pending"), (prev, "prev"), (pos_base, "pos_base")):
        _expect(t, torch.int32, (b * c,), name)
    if draft_tokens is not None and (draft_tokens.dtype != torch.int32 or draft_tokens.numel() != kd * b * c):
        raise ValueError("draft_tokens must be int32 [kd][b][c]")
    cap = 0
    if out_tokens is not None:
        if out_tokens.dtype != torch.int32 or out_tokens.dim() != 2 or out_tokens.shape[0] != b:
            raise ValueError("out_tokens must be int32 [b][capacity]")
        cap = out_tokens.shape[1]
        _expect(out_len, torch.int32, (b,), "out_len")
    _check(load().sq_spec_commit_multi(_ptr(n_accepted), _ptr(next_token), _ptr(chain), _ptr(draft_tokens), b, c, kd,
                                       _ptr(pending), _ptr(prev), _ptr(pos_base), _ptr(out_tokens), cap, _ptr(out_len),
                                       _ptr(status), _stream(n_accepted.device)), "sq_spec_commit_multi")
