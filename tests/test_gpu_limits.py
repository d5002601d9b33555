"""GPU parity at the largest sizes each call accepts, and at the degenerate
ends of its ranges, against the CPU oracle."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_21704_amd as sq
from accept_compare import check_accept
from paper_2609_21704_amd import synth

pytestmark = pytest.mark.gpu
DEV = "cuda"
GEMV_TOL = 2e-3
KMAX = 1 << 20


def bits16(t: torch.Tensor) -> np.ndarray:
    return t.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)


@pytest.mark.parametrize("m", [1, 8])
def test_qgemv_w4a16_longest_k(m):
    n = 3
    w = synth.normal_f16((n, KMAX), 0.02, synth.stream_seed(31, m))
    x = synth.normal_f16((m, KMAX), 1.0, synth.stream_seed(32, m))
    codes, scales, zeros = sq.sq_quantize_int4_g128(w.to(DEV))
    c_ref, s_ref, z_ref = oracle.quantize_int4_g128(bits16(w))
    assert np.array_equal(codes.cpu().numpy(), c_ref)
    y_ref, d_ref = oracle.qgemv_w4a16(bits16(x), c_ref, s_ref, z_ref)
    y = sq.sq_qgemv_w4a16(x.to(DEV), codes, scales, zeros, y_dtype=torch.float32)
    assert oracle.normalised_error(y.cpu().numpy(), y_ref, d_ref) <= GEMV_TOL


@pytest.mark.parametrize("m", [1, 8])
def test_qgemv_w8a16_longest_k(m):
    n = 3
    w = synth.normal_f16((n, KMAX), 0.02, synth.stream_seed(33, m))
    x = synth.normal_f16((m, KMAX), 1.0, synth.stream_seed(34, m))
    codes, scales = sq.sq_quantize_fp8_e4m3(w.to(DEV))
    c_ref, s_ref = oracle.quantize_fp8_e4m3(bits16(w))
    assert np.array_equal(codes.cpu().numpy(), c_ref)
    y_ref, d_ref = oracle.qgemv_w8a16(bits16(x), c_ref, s_ref)
    y = sq.sq_qgemv_w8a16(x.to(DEV), codes, scales, y_dtype=torch.float32)
    assert oracle.normalised_error(y.cpu().numpy(), y_ref, d_ref) <= GEMV_TOL


def test_verify_gemm_longest_k_and_most_rows():
    m, n = 64, 17
    w = synth.normal_f16((n, KMAX), 0.02, 35)
    x = synth.normal_f16((m, KMAX), 1.0, 36)
    y_ref, d_ref = oracle.gemm_f16(bits16(x), bits16(w))
    y = sq.sq_verify_gemm_f16(x.to(DEV), w.to(DEV), y_dtype=torch.float32)
    assert oracle.normalised_error(y.cpu().numpy(), y_ref, d_ref) <= GEMV_TOL


def test_spec_accept_largest_vocabulary():
    b, kd, v = 1, 1, 1 << 26
    draft = synth.normal_f32((kd, b, v), 2.0, 37)
    target = synth.normal_f32((b, kd + 1, v), 2.0, 38)
    target[:, :kd] += draft.permute(1, 0, 2)
    tok = torch.tensor([[v - 5]], dtype=torch.int32)
    q_out = torch.empty((kd, b, v), dtype=torch.float32, device=DEV)
    p_out = torch.empty((b, kd + 1, v), dtype=torch.float32, device=DEV)
    for u in (0, 1 << 23, (1 << 24) - 1):
        u24 = torch.tensor([[u, (u * 7 + 12345) & 0xFFFFFF]], dtype=torch.int32)
        n, t = sq.sq_spec_accept(draft.to(DEV), target.to(DEV), tok.to(DEV), u24.to(DEV), 1.0,
                                 q_out=q_out, p_out=p_out)
        check_accept(draft.numpy(), target.numpy(), tok.numpy(), u24.numpy(), 1.0, n.cpu().numpy(),
                     t.cpu().numpy(), q_out.cpu().numpy(), p_out.cpu().numpy())


def test_spec_accept_most_sequences():
    b, kd, v = (1 << 24) - 1, 0, 3
    target = synth.normal_f32((b, 1, v), 2.0, 39)
    u24 = synth.uniform_u24((b, 1), 40)
    p_out = torch.empty((b, 1, v), dtype=torch.float32, device=DEV)
    n, t = sq.sq_spec_accept(None, target.to(DEV), None, u24.to(DEV), 1.0, p_out=p_out)
    check_accept(None, target.numpy(), np.zeros((0, b), np.int32), u24.numpy(), 1.0, n.cpu().numpy(),
                 t.cpu().numpy(), None, p_out.cpu().numpy())


@pytest.mark.parametrize("temp", [1.0, 0.0])
def test_spec_accept_single_token_vocabulary(temp):
    b, kd, v = 3, 2, 1
    draft = synth.normal_f32((kd, b, v), 2.0, 41)
    target = synth.normal_f32((b, kd + 1, v), 2.0, 42)
    tok = torch.zeros((kd, b), dtype=torch.int32)
    u24 = synth.uniform_u24((b, kd + 1), 43)
    n, t = sq.sq_spec_accept(draft.to(DEV), target.to(DEV), tok.to(DEV), u24.to(DEV), temp)
    assert np.all(n.cpu().numpy() == kd) and np.all(t.cpu().numpy() == 0)
