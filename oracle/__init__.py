"""SpecQuant CPU oracle -- test infrastructure only.

A plain fp64 C implementation (``sq_oracle.c``; ``sq_decoder.c`` for the
operations of the decoder layer around the projections; ``sq_multi.c`` for
the acceptance of several draft chains per sequence) of what the SpecQuant
hot path computes, wrapped with ctypes for numpy arrays; ``decoder.py``
composes them into the decoder and the speculative round with its cache.  Only the test suite,
``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py`` may use
it; the product path (the HIP library and its binding) never imports it, and
it imports nothing from the product path.

Paper: SpecQuant (arXiv 2609.21704): quantized parents Q4 = f(W16, 4) and
Q8 = f(W16, 8) (SS III-A.1, III-A.2), the parent Q16 = W16 (SS III-A.3), draft
generation (SS III-D.2), parent verification (SS III-D.3) and token acceptance
or correction (SS III-D.4, guess-set rule of SS III-A).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRCS = [os.path.join(_HERE, f) for f in ("sq_oracle.c", "sq_decoder.c", "sq_multi.c")]
_LIB_PATH = os.path.join(_HERE, "libsq_oracle.so")
_lib = None

OK, ERR_NULL, ERR_SHAPE, ERR_NONFINITE, ERR_VALUE = 0, 1, 2, 5, 6


def build(force: bool = True) -> str:
    """Compile the oracle with gcc: fp64, no contraction, no fast-math, OpenMP."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp"
        cmd = ["gcc", "-std=c11", "-O2", "-fopenmp", "-ffp-contract=off", "-fno-fast-math",
               "-fPIC", "-shared", "-Wall", *_SRCS, "-o", tmp, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        build(force=True)
    lib = ctypes.CDLL(_LIB_PATH)
    P = ctypes.c_void_p
    I64 = ctypes.c_int64
    I32 = ctypes.c_int32
    D = ctypes.c_double
    sigs = {
        "sqo_num_threads": ([], ctypes.c_int),
        "sqo_set_num_threads": ([ctypes.c_int], None),
        "sqo_f16_to_f64": ([ctypes.c_uint16], D),
        "sqo_f16_round_up": ([D], D),
        "sqo_fp8_e4m3_decode": ([ctypes.c_uint8], D),
        "sqo_fp8_e4m3_encode": ([D], ctypes.c_uint8),
        "sqo_quantize_int4_g128": ([P, I64, I64, P, P, P], ctypes.c_int),
        "sqo_dequant_int4": ([P, P, P, I64, I64, P], ctypes.c_int),
        "sqo_quantize_fp8_e4m3": ([P, I64, I64, P, P], ctypes.c_int),
        "sqo_dequant_fp8": ([P, P, I64, I64, P], ctypes.c_int),
        "sqo_qgemv_w4a16": ([P, I64, I64, P, P, P, I64, P, P], ctypes.c_int),
        "sqo_qgemv_w8a16": ([P, I64, I64, P, P, I64, P, P], ctypes.c_int),
        "sqo_gemm_f16": ([P, I64, I64, P, I64, P, P], ctypes.c_int),
        "sqo_softmax": ([P, I64, I64, D, P], ctypes.c_int),
        "sqo_spec_accept": ([P, P, P, P, I32, I32, I32, D, P, P, P, P], ctypes.c_int),
        "sqo_accept_probs": ([P, P, P, P, I32, I32, I32, P, P], ctypes.c_int),
        "sqo_rmsnorm": ([P, I64, I64, P, D, P], ctypes.c_int),
        "sqo_rope": ([P, I64, I64, I64, P, D], ctypes.c_int),
        "sqo_attention": ([P, I64, I64, I64, I64, P, P, I64, P, P], ctypes.c_int),
        "sqo_silu_mul": ([P, I64, I64, P], ctypes.c_int),
        "sqo_multi_accept_probs": ([P, P, P, P, I32, I32, I32, I32, P, P, P], ctypes.c_int),
        "sqo_multi_accept_greedy": ([P, P, I32, I32, I32, I32, P, P, P], ctypes.c_int),
    }
    for name, (args, res) in sigs.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = res
    _lib = lib
    return lib


def _ptr(a):
    return None if a is None else a.ctypes.data


def _f16_bits(a) -> np.ndarray:
    a = np.asarray(a)
    if a.dtype == np.float16:
        a = a.view(np.uint16)
    if a.dtype != np.uint16:
        raise TypeError("expected float16 values or their uint16 bit patterns")
    return np.ascontiguousarray(a)


def _check(status: int, what: str):
    if status != OK:
        raise OracleError(status, what)


class OracleError(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__(f"{what}: oracle status {status}")
        self.status = status


def num_threads() -> int:
    return int(_load().sqo_num_threads())


def set_num_threads(n: int) -> None:
    """Threads of later oracle calls (timing only: the results do not depend on it)."""
    _load().sqo_set_num_threads(int(n))


# ------------------------------------------------------------ scalar helpers
def f16_to_f64(bits: int) -> float:
    return float(_load().sqo_f16_to_f64(int(bits)))


def f16_round_up(s: float) -> float:
    """Smallest binary16 value >= s (s finite, > 0)."""
    return float(_load().sqo_f16_round_up(float(s)))


def fp8_decode(code: int) -> float:
    return float(_load().sqo_fp8_e4m3_decode(int(code)))


def fp8_encode(v: float) -> int:
    return int(_load().sqo_fp8_e4m3_encode(float(v)))


# --------------------------------------------------------------- quantizers
def quantize_int4_g128(w):
    """Q4 = f(W16, 4): returns (codes u8 [n][k/2], scales f16-bits [n][k/128],
    zeros f16-bits [n][k/128])."""
    w = _f16_bits(w)
    n, k = w.shape
    codes = np.zeros((n, k // 2), np.uint8)
    scales = np.zeros((n, max(k // 128, 1)), np.uint16)
    zeros = np.zeros((n, max(k // 128, 1)), np.uint16)
    _check(_load().sqo_quantize_int4_g128(_ptr(w), n, k, _ptr(codes), _ptr(scales), _ptr(zeros)),
           "quantize_int4_g128")
    return codes, scales, zeros


def dequant_int4(codes, scales, zeros, k: int) -> np.ndarray:
    codes = np.ascontiguousarray(codes, np.uint8)
    scales, zeros = _f16_bits(scales), _f16_bits(zeros)
    n = codes.shape[0]
    out = np.zeros((n, k), np.float64)
    _check(_load().sqo_dequant_int4(_ptr(codes), _ptr(scales), _ptr(zeros), n, k, _ptr(out)), "dequant_int4")
    return out


def quantize_fp8_e4m3(w):
    """Q8 = f(W16, 8): returns (codes u8 [n][k], scales f32 [n])."""
    w = _f16_bits(w)
    n, k = w.shape
    codes = np.zeros((n, k), np.uint8)
    scales = np.zeros((n,), np.float32)
    _check(_load().sqo_quantize_fp8_e4m3(_ptr(w), n, k, _ptr(codes), _ptr(scales)), "quantize_fp8_e4m3")
    return codes, scales


def dequant_fp8(codes, scales) -> np.ndarray:
    codes = np.ascontiguousarray(codes, np.uint8)
    scales = np.ascontiguousarray(scales, np.float32)
    n, k = codes.shape
    out = np.zeros((n, k), np.float64)
    _check(_load().sqo_dequant_fp8(_ptr(codes), _ptr(scales), n, k, _ptr(out)), "dequant_fp8")
    return out


# ---------------------------------------------------------- GEMV and GEMM
def qgemv_w4a16(x, codes, scales, zeros):
    """fp64 y = x . W'^T and normaliser d = sum |x * W'| for INT4 g128 W'."""
    x = _f16_bits(np.atleast_2d(x))
    codes = np.ascontiguousarray(codes, np.uint8)
    scales, zeros = _f16_bits(scales), _f16_bits(zeros)
    m, k = x.shape
    n = codes.shape[0]
    y = np.zeros((m, n), np.float64)
    d = np.zeros((m, n), np.float64)
    _check(_load().sqo_qgemv_w4a16(_ptr(x), m, k, _ptr(codes), _ptr(scales), _ptr(zeros), n, _ptr(y), _ptr(d)),
           "qgemv_w4a16")
    return y, d


def qgemv_w8a16(x, codes, scales):
    x = _f16_bits(np.atleast_2d(x))
    codes = np.ascontiguousarray(codes, np.uint8)
    scales = np.ascontiguousarray(scales, np.float32)
    m, k = x.shape
    n = codes.shape[0]
    y = np.zeros((m, n), np.float64)
    d = np.zeros((m, n), np.float64)
    _check(_load().sqo_qgemv_w8a16(_ptr(x), m, k, _ptr(codes), _ptr(scales), n, _ptr(y), _ptr(d)), "qgemv_w8a16")
    return y, d


def gemm_f16(x, w):
    x = _f16_bits(np.atleast_2d(x))
    w = _f16_bits(w)
    m, k = x.shape
    n = w.shape[0]
    y = np.zeros((m, n), np.float64)
    d = np.zeros((m, n), np.float64)
    _check(_load().sqo_gemm_f16(_ptr(x), m, k, _ptr(w), n, _ptr(y), _ptr(d)), "gemm_f16")
    return y, d


# ------------------------------------------------------- softmax / accept
def softmax(logits, temperature: float = 1.0) -> np.ndarray:
    logits = np.ascontiguousarray(np.atleast_2d(logits), np.float32)
    rows, v = logits.shape
    p = np.zeros((rows, v), np.float64)
    _check(_load().sqo_softmax(_ptr(logits), rows, v, float(temperature), _ptr(p)), "softmax")
    return p


def spec_accept(draft_logits, target_logits, draft_tokens, u24, temperature: float = 1.0,
                want_pq: bool = False):
    """Speculative accept / resample.

    draft_logits [kd][b][v] f32, target_logits [b][kd+1][v] f32,
    draft_tokens [kd][b] i32, u24 [b][kd+1] u32 (low 24 bits used).
    Returns (n_accepted [b], next_token [b], q [kd][b][v] | None, p [b][kd+1][v] | None);
    q and p are the fp64 distributions (the decisions use their fp32 roundings).
    A sequence with a row that has no distribution (a NaN or +inf logit, or no
    finite logit) gets n_accepted = next_token = -1.
    """
    target_logits = np.ascontiguousarray(target_logits, np.float32)
    b, kd1, v = target_logits.shape
    kd = kd1 - 1
    if kd > 0:
        draft_logits = np.ascontiguousarray(draft_logits, np.float32).reshape(kd, b, v)
        draft_tokens = np.ascontiguousarray(draft_tokens, np.int32).reshape(kd, b)
    else:
        draft_logits = None
        draft_tokens = None
    u24 = None if u24 is None else np.ascontiguousarray(u24, np.uint32).reshape(b, kd + 1)
    n_acc = np.zeros(b, np.int32)
    nxt = np.zeros(b, np.int32)
    q = np.zeros((max(kd, 1), b, v), np.float64) if want_pq and kd > 0 else None
    p = np.zeros((b, kd + 1, v), np.float64) if want_pq else None
    _check(_load().sqo_spec_accept(_ptr(draft_logits), _ptr(target_logits), _ptr(draft_tokens), _ptr(u24),
                                   b, kd, v, float(temperature), _ptr(n_acc), _ptr(nxt), _ptr(q), _ptr(p)),
           "spec_accept")
    return n_acc, nxt, q, p


def accept_probs(p, q, draft_tokens, u24):
    """The decisions and draws of spec_accept (T > 0) from given fp32
    distributions: p [b][kd+1][v] f32, q [kd][b][v] f32 (None when kd = 0),
    draft_tokens [kd][b] i32, u24 [b][kd+1] u32.  Returns (n_accepted [b],
    next_token [b])."""
    p = np.ascontiguousarray(p, np.float32)
    b, kd1, v = p.shape
    kd = kd1 - 1
    if kd > 0:
        q = np.ascontiguousarray(q, np.float32).reshape(kd, b, v)
        draft_tokens = np.ascontiguousarray(draft_tokens, np.int32).reshape(kd, b)
    else:
        q = draft_tokens = None
    u24 = np.ascontiguousarray(u24, np.uint32).reshape(b, kd + 1)
    n_acc = np.zeros(b, np.int32)
    nxt = np.zeros(b, np.int32)
    _check(_load().sqo_accept_probs(_ptr(p), _ptr(q), _ptr(draft_tokens), _ptr(u24), b, kd, v, _ptr(n_acc),
                                    _ptr(nxt)), "accept_probs")
    return n_acc, nxt


def multi_accept_probs(p, q, drafts, u24):
    """Multi-candidate acceptance (recursive rejection over c draft chains)
    from fp32 distributions: p [b][c][kd+1][v], q [kd][b][c][v],
    drafts [kd][b][c] i32, u24 [b][c kd + 1].  Returns (n_accepted [b],
    next_token [b], chain [b])."""
    p = np.ascontiguousarray(p, np.float32)
    b, c, kd1, v = p.shape
    kd = kd1 - 1
    if kd > 0:
        q = np.ascontiguousarray(q, np.float32).reshape(kd, b, c, v)
        drafts = np.ascontiguousarray(drafts, np.int32).reshape(kd, b, c)
    else:
        q = drafts = None
    u24 = np.ascontiguousarray(u24, np.uint32).reshape(b, c * kd + 1)
    n = np.zeros(b, np.int32)
    t = np.zeros(b, np.int32)
    ch = np.zeros(b, np.int32)
    _check(_load().sqo_multi_accept_probs(_ptr(p), _ptr(q), _ptr(drafts), _ptr(u24), b, c, kd, v, _ptr(n), _ptr(t),
                                          _ptr(ch)), "multi_accept_probs")
    return n, t, ch


def multi_accept_greedy(target_logits, drafts):
    """Greedy multi-candidate acceptance from target logits [b][c][kd+1][v]
    and drafts [kd][b][c].  Returns (n_accepted, next_token, chain)."""
    target_logits = np.ascontiguousarray(target_logits, np.float32)
    b, c, kd1, v = target_logits.shape
    kd = kd1 - 1
    drafts = None if kd == 0 else np.ascontiguousarray(drafts, np.int32).reshape(kd, b, c)
    n = np.zeros(b, np.int32)
    t = np.zeros(b, np.int32)
    ch = np.zeros(b, np.int32)
    _check(_load().sqo_multi_accept_greedy(_ptr(target_logits), _ptr(drafts), b, c, kd, v, _ptr(n), _ptr(t), _ptr(ch)),
           "multi_accept_greedy")
    return n, t, ch


def multi_accept(draft_logits, target_logits, drafts, u24, temperature: float = 1.0):
    """Multi-candidate acceptance from logits: draft_logits [kd][b][c][v],
    target_logits [b][c][kd+1][v]; T > 0: the distributions are fp64
    softmaxes held in fp32, then multi_accept_probs; T = 0: greedy."""
    target_logits = np.ascontiguousarray(target_logits, np.float32)
    b, c, kd1, v = target_logits.shape
    kd = kd1 - 1
    if temperature == 0.0:
        return multi_accept_greedy(target_logits, drafts)
    p = softmax(target_logits.reshape(-1, v), temperature).astype(np.float32).reshape(b, c, kd1, v)
    q = None
    if kd > 0:
        q = softmax(np.ascontiguousarray(draft_logits, np.float32).reshape(-1, v), temperature)
        q = q.astype(np.float32).reshape(kd, b, c, v)
    return multi_accept_probs(p, q, drafts, u24)


def rmsnorm(h, w, eps: float) -> np.ndarray:
    """y = h / sqrt(mean(h^2) + eps) * w per row, fp64 (h [m][d], w [d])."""
    h = np.ascontiguousarray(np.atleast_2d(h), np.float64)
    m, d = h.shape
    w = np.ascontiguousarray(w, np.float64).reshape(d)
    y = np.zeros((m, d), np.float64)
    _check(_load().sqo_rmsnorm(_ptr(h), m, d, _ptr(w), float(eps), _ptr(y)), "rmsnorm")
    return y


def rope(x, pos, theta: float) -> np.ndarray:
    """Rotary embedding of x [n][heads][hd] at positions pos [n] (returns a new array)."""
    x = np.array(x, np.float64, order="C", copy=True)
    n, heads, hd = x.shape
    pos = np.ascontiguousarray(pos, np.int64).reshape(n)
    _check(_load().sqo_rope(_ptr(x), n, heads, hd, _ptr(pos), float(theta)), "rope")
    return x


def attention(q, kc, vc, pos) -> np.ndarray:
    """Causal GQA attention of one sequence: q [n][hq][hd], kc / vc [hkv][len][hd],
    row i attends to positions 0 .. pos[i].  Returns [n][hq][hd] fp64."""
    q = np.ascontiguousarray(q, np.float64)
    kc = np.ascontiguousarray(kc, np.float64)
    vc = np.ascontiguousarray(vc, np.float64)
    n, hq, hd = q.shape
    hkv, length, hd2 = kc.shape
    if vc.shape != kc.shape or hd2 != hd:
        raise ValueError("attention: cache shapes do not match")
    pos = np.ascontiguousarray(pos, np.int64).reshape(n)
    out = np.zeros((n, hq, hd), np.float64)
    _check(_load().sqo_attention(_ptr(q), n, hq, hkv, hd, _ptr(kc), _ptr(vc), length, _ptr(pos), _ptr(out)),
           "attention")
    return out


def silu_mul(gu) -> np.ndarray:
    """g / (1 + exp(-g)) * u with gate | up = the two halves of each row of gu [m][2 I]."""
    gu = np.ascontiguousarray(np.atleast_2d(gu), np.float64)
    m, two_i = gu.shape
    out = np.zeros((m, two_i // 2), np.float64)
    _check(_load().sqo_silu_mul(_ptr(gu), m, two_i // 2, _ptr(out)), "silu_mul")
    return out


def normalised_error(y_test, y_ref, d_ref) -> float:
    """max |y_test - y_ref| / d over all outputs; d = sum |x * w'| per output.
    Where d == 0 the output must be exactly zero (returns inf otherwise)."""
    y_test = np.asarray(y_test, np.float64)
    err = np.abs(y_test - y_ref)
    zero = d_ref == 0
    if np.any(err[zero] != 0):
        return float("inf")
    if np.all(zero):
        return 0.0
    return float(np.max(err[~zero] / d_ref[~zero]))
