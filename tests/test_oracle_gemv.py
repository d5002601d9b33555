"""Pins of the oracle's GEMV/GEMM (draft pass on Q4/Q8 and verify pass on
Q16 = W16; SpecQuant SS III-D.2, III-D.3) against numpy matmul on weights
decoded here, and closed forms (identity, unit vectors, row sums)."""
import numpy as np

import oracle

RNG = np.random.default_rng(99)


def _f16(a):
    return np.asarray(a, np.float64).astype(np.float16)


def _np_dequant_int4(codes, scales, zeros, k):
    n = codes.shape[0]
    q = np.empty((n, k), np.float64)
    q[:, 0::2] = codes & 15
    q[:, 1::2] = codes >> 4
    s = np.repeat(scales.view(np.float16).astype(np.float64), 128, axis=1)
    z = np.repeat(zeros.view(np.float16).astype(np.float64), 128, axis=1)
    return (q - z) * s


def _np_dequant_fp8(codes, scales):
    import torch
    table = torch.arange(256, dtype=torch.int32).to(torch.uint8).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    return table[codes] * scales.astype(np.float64)[:, None]


def test_w4a16_matches_numpy_matmul():
    m, k, n = 3, 384, 37
    w = _f16(RNG.normal(0, 0.02, (n, k)))
    x = _f16(RNG.normal(0, 1, (m, k)))
    codes, scales, zeros = oracle.quantize_int4_g128(w)
    y, d = oracle.qgemv_w4a16(x, codes, scales, zeros)
    wd = _np_dequant_int4(codes, scales, zeros, k)
    x64 = x.astype(np.float64)
    assert np.allclose(y, x64 @ wd.T, rtol=0, atol=1e-12)
    assert np.allclose(d, np.abs(x64) @ np.abs(wd).T, rtol=1e-13, atol=0)


def test_w8a16_matches_numpy_matmul():
    m, k, n = 4, 272, 29
    w = _f16(RNG.normal(0, 0.02, (n, k)))
    x = _f16(RNG.normal(0, 1, (m, k)))
    codes, scales = oracle.quantize_fp8_e4m3(w)
    y, d = oracle.qgemv_w8a16(x, codes, scales)
    wd = _np_dequant_fp8(codes, scales)
    x64 = x.astype(np.float64)
    assert np.allclose(y, x64 @ wd.T, rtol=0, atol=1e-12)
    assert np.allclose(d, np.abs(x64) @ np.abs(wd).T, rtol=1e-13, atol=0)


def test_gemm_f16_matches_numpy_and_rows_equal_gemv():
    m, k, n = 7, 200, 41
    w = _f16(RNG.normal(0, 0.02, (n, k)))
    x = _f16(RNG.normal(0, 1, (m, k)))
    y, d = oracle.gemm_f16(x, w)
    x64, w64 = x.astype(np.float64), w.astype(np.float64)
    assert np.allclose(y, x64 @ w64.T, rtol=0, atol=1e-12)
    for i in range(m):
        yi, _ = oracle.gemm_f16(x[i:i + 1], w)
        assert np.array_equal(yi[0], y[i])


def test_identity_and_unit_vector_closed_forms():
    k = 256
    eye = np.eye(k, dtype=np.float16)
    x = _f16(RNG.normal(0, 1, (2, k)))
    # Q16 = W16 identity: y = x exactly
    y, _ = oracle.gemm_f16(x, eye)
    assert np.array_equal(y, x.astype(np.float64))
    # INT4 identity: each row's nonzero group is a one-hot group -> 1.00067138671875 * x
    codes, scales, zeros = oracle.quantize_int4_g128(eye)
    y4, _ = oracle.qgemv_w4a16(x, codes, scales, zeros)
    assert np.array_equal(y4, 1.00067138671875 * x.astype(np.float64))
    # FP8 identity: amax = 1 -> s = 1/448 (fp32), code(448) -> w' = 448 * fl32(1/448)
    c8, s8 = oracle.quantize_fp8_e4m3(eye)
    y8, _ = oracle.qgemv_w8a16(x, c8, s8)
    assert np.array_equal(y8, 448.0 * float(np.float32(1.0 / 448.0)) * x.astype(np.float64))
    # unit vector e_j picks column j of W'; all-ones x gives row sums
    n = 19
    w = _f16(RNG.normal(0, 0.02, (n, k)))
    codes, scales, zeros = oracle.quantize_int4_g128(w)
    wd = _np_dequant_int4(codes, scales, zeros, k)
    for j in (0, 1, 127, 128, 255):
        e = np.zeros((1, k), np.float16)
        e[0, j] = 1
        yj, _ = oracle.qgemv_w4a16(e, codes, scales, zeros)
        assert np.array_equal(yj[0], wd[:, j])
    ones = np.ones((1, k), np.float16)
    yo, _ = oracle.gemm_f16(ones, w)
    assert np.allclose(yo[0], w.astype(np.float64).sum(axis=1), rtol=0, atol=1e-15)


def test_normalised_error_metric():
    y_ref = np.array([[1.0, 0.0]])
    d_ref = np.array([[2.0, 0.0]])
    assert abs(oracle.normalised_error(np.array([[1.002, 0.0]]), y_ref, d_ref) - 0.001) < 1e-15
    assert oracle.normalised_error(np.array([[1.0, 1e-30]]), y_ref, d_ref) == float("inf")


def test_results_do_not_depend_on_the_thread_count():
    rng = np.random.default_rng(7)
    w = _f16(rng.normal(0, 0.02, (300, 512)))
    x = _f16(rng.normal(0, 1, (3, 512)))
    c, sc, z = oracle.quantize_int4_g128(w)
    n = oracle.num_threads()
    try:
        oracle.set_num_threads(1)
        one = (oracle.qgemv_w4a16(x, c, sc, z)[0], oracle.gemm_f16(x, w)[0])
        oracle.set_num_threads(max(2, n))
        many = (oracle.qgemv_w4a16(x, c, sc, z)[0], oracle.gemm_f16(x, w)[0])
    finally:
        oracle.set_num_threads(n)
    for a, b in zip(one, many):
        assert np.array_equal(a, b)
