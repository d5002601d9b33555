"""GPU parity on seeded random shapes: every GEMV / verify entry point against
the CPU oracle at (m, n, k) drawn from a fixed seed, so that the dispatch
rules (row blocks, tasks of rows, K slices, the matrix-core kernels) and the
ragged ends of each kernel meet shapes nobody picked by hand.  Same bar as
the hand-picked cases: max |y - y_ref| / sum |x w'| <= 2e-3."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_21704_amd as sq
from paper_2609_21704_amd import synth

pytestmark = pytest.mark.gpu
DEV = "cuda"
GEMV_TOL = 2e-3


def bits16(t: torch.Tensor) -> np.ndarray:
    return t.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)


def _shapes(seed, count, m_max, k_unit, k_units_max, n_max=6000, weights_max=24_000_000, n_min=1, k_units_min=1):
    """(m, n, k): n log-uniform in [n_min, n_max], k a multiple of k_unit, at
    most weights_max weights, so that the oracle finishes in about a second."""
    rng = np.random.default_rng(seed)
    out = []
    while len(out) < count:
        m = int(rng.integers(1, m_max + 1))
        n = int(np.exp(rng.uniform(np.log(n_min), np.log(n_max))))
        k = k_unit * int(rng.integers(k_units_min, k_units_max + 1))
        if n * k <= weights_max:
            out.append((m, max(n, 1), k))
    return out


W4_SHAPES = _shapes(101, 12, 8, 128, 120)
# many rows of 2048 .. 4096 k at m <= 2: row blocks of many rows, three rows a step
W4_SHAPES += _shapes(105, 6, 2, 128, 32, n_min=1000, n_max=40000, k_units_min=16)
W8_SHAPES = _shapes(102, 10, 8, 16, 1200)
F16_SHAPES = _shapes(103, 12, 64, 8, 2500)
# small m (the row-block kernels) more often, and many rows
F16_SHAPES += _shapes(104, 8, 8, 16, 1200)
F16_SHAPES += _shapes(106, 6, 8, 16, 256, n_min=1000, n_max=40000, k_units_min=32)


def _inputs(m, n, k, seed):
    w = synth.normal_f16((n, k), 0.02, synth.stream_seed(seed, 1, n, k))
    x = synth.normal_f16((m, k), 1.0, synth.stream_seed(seed, 2, m, k))
    return w, x


@pytest.mark.parametrize("m,n,k", W4_SHAPES)
def test_qgemv_w4a16_random_shape(m, n, k):
    w, x = _inputs(m, n, k, 61)
    codes, scales, zeros = sq.sq_quantize_int4_g128(w.to(DEV))
    c_ref, s_ref, z_ref = oracle.quantize_int4_g128(bits16(w))
    assert np.array_equal(codes.cpu().numpy(), c_ref)
    y_ref, d_ref = oracle.qgemv_w4a16(bits16(x), c_ref, s_ref, z_ref)
    y = sq.sq_qgemv_w4a16(x.to(DEV), codes, scales, zeros, y_dtype=torch.float32)
    assert oracle.normalised_error(y.cpu().numpy(), y_ref, d_ref) <= GEMV_TOL


@pytest.mark.parametrize("m,n,k", W8_SHAPES)
def test_qgemv_w8a16_random_shape(m, n, k):
    w, x = _inputs(m, n, k, 62)
    codes, scales = sq.sq_quantize_fp8_e4m3(w.to(DEV))
    c_ref, s_ref = oracle.quantize_fp8_e4m3(bits16(w))
    assert np.array_equal(codes.cpu().numpy(), c_ref)
    y_ref, d_ref = oracle.qgemv_w8a16(bits16(x), c_ref, s_ref)
    y = sq.sq_qgemv_w8a16(x.to(DEV), codes, scales, y_dtype=torch.float32)
    assert oracle.normalised_error(y.cpu().numpy(), y_ref, d_ref) <= GEMV_TOL


@pytest.mark.parametrize("m,n,k", F16_SHAPES)
def test_verify_gemm_f16_random_shape(m, n, k):
    w, x = _inputs(m, n, k, 63)
    y_ref, d_ref = oracle.gemm_f16(bits16(x), bits16(w))
    y = sq.sq_verify_gemm_f16(x.to(DEV), w.to(DEV), y_dtype=torch.float32)
    assert oracle.normalised_error(y.cpu().numpy(), y_ref, d_ref) <= GEMV_TOL
