"""Pins of the oracle's quantizers (Q4 = f(W16,4), Q8 = f(W16,8); SpecQuant
SS III-A.1, III-A.2) against facts that do not come from the oracle itself:
numpy's binary16 arithmetic, torch's float8_e4m3fn conversion, brute-force
nearest-grid searches written here, and closed forms."""
import numpy as np
import pytest
import torch

import oracle

RNG = np.random.default_rng(1234)


# ------------------------------------------------------------------ fp16 ----
def test_f16_decode_all_patterns_match_numpy():
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    ref = bits.view(np.float16).astype(np.float64)
    got = np.array([oracle.f16_to_f64(int(b)) for b in bits])
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], ref[~nan])
    # signed zero kept
    assert np.signbit(got[0x8000]) and not np.signbit(got[0])


def _numpy_round_up_f16(s: float) -> float:
    h = np.float16(s)  # numpy converts float64 -> float16 with round-to-nearest-even
    if float(h) < s:
        h = np.nextafter(h, np.float16(np.inf))
    return float(h)


def test_f16_round_up_matches_numpy_nextafter():
    vals = np.concatenate([
        np.exp(RNG.uniform(np.log(1e-8), np.log(6e4), 20000)),
        [2.0 ** -24, 2.0 ** -14, 2.0 ** -14 * 1.0001, 1.0, 1.0 + 2 ** -11, 1.0 + 2 ** -10, 65504.0 - 1e-9],
        (np.arange(1, 2000) / 15.0) * 2.0 ** -10,
    ])
    for s in vals:
        assert oracle.f16_round_up(float(s)) == _numpy_round_up_f16(float(s)), s


# ------------------------------------------------------------------ INT4 ----
def _groups_under_test():
    k = 128 * 6
    rows = [
        RNG.normal(0, 0.02, k),                       # the configs' weight law
        RNG.normal(0, 1.0, k),
        RNG.uniform(0.1, 2.0, k),                     # all positive: lo clamps to 0
        -RNG.uniform(0.1, 2.0, k),                    # all negative: hi clamps to 0
        RNG.standard_t(2, k) * 0.05,                  # heavy tails
        RNG.normal(0, 1e-6, k),                       # fp16 subnormal range
        np.full(k, 0.3),                              # constant positive
        np.r_[np.zeros(k // 2), RNG.normal(0, 3, k // 2)],
    ]
    w = np.stack(rows).astype(np.float16)
    w[7, 130] = np.float16(-0.0)
    return w


def _decode_int4(codes, scales, zeros, k):
    n = codes.shape[0]
    q = np.empty((n, k), np.int64)
    q[:, 0::2] = codes & 15
    q[:, 1::2] = codes >> 4
    s = np.repeat(scales.view(np.float16).astype(np.float64), 128, axis=1)
    z = np.repeat(zeros.view(np.float16).astype(np.float64), 128, axis=1)
    return q, s, z


def test_int4_half_step_invariant_and_grid():
    w = _groups_under_test()
    n, k = w.shape
    codes, scales, zeros = oracle.quantize_int4_g128(w)
    q, s, z = _decode_int4(codes, scales, zeros, k)
    w64 = w.astype(np.float64)
    wd = (q - z) * s
    # |w - w'| <= s/2 for every element
    assert np.all(np.abs(w64 - wd) <= s / 2)
    # zero points are integers in [0, 15]; codes in [0, 15]
    assert np.all(z == np.round(z)) and z.min() >= 0 and z.max() <= 15
    # scale = smallest fp16 >= (hi - lo)/15 with the range widened to contain 0
    g = w64.reshape(n, k // 128, 128)
    lo = np.minimum(g.min(axis=2), 0.0)
    hi = np.maximum(g.max(axis=2), 0.0)
    sc = scales.view(np.float16).astype(np.float64)
    for (r, j), val in np.ndenumerate(sc):
        if hi[r, j] == lo[r, j]:
            assert val == 1.0
        else:
            assert val == _numpy_round_up_f16((hi[r, j] - lo[r, j]) / 15.0)


def test_int4_codes_are_brute_force_nearest_with_ties_to_even():
    w = _groups_under_test()
    n, k = w.shape
    codes, scales, zeros = oracle.quantize_int4_g128(w)
    q, s, z = _decode_int4(codes, scales, zeros, k)
    w64 = w.astype(np.float64)
    # candidate offsets r = c - z for every code c in 0..15
    cand = np.arange(16)[None, None, :] - z[:, :, None]           # [n][k][16]
    dist = np.abs(w64[:, :, None] - cand * s[:, :, None])         # exact in fp64
    best = dist.min(axis=2, keepdims=True)
    ties = dist == best
    # among the nearest codes, pick the one whose offset (c - z) is even
    even = (cand % 2 == 0)
    pick = np.where(ties.sum(axis=2) > 1, np.argmax(ties & even, axis=2), np.argmax(ties, axis=2))
    assert np.array_equal(pick, q)


def test_int4_closed_forms():
    k = 256
    # one 1 among zeros (group 0), all-zero group 1
    w = np.zeros((1, k), np.float16)
    w[0, 5] = 1.0
    codes, scales, zeros = oracle.quantize_int4_g128(w)
    s = scales.view(np.float16).astype(np.float64)[0]
    assert s[0] == 1093 * 2.0 ** -14 == 0.06671142578125
    assert s[1] == 1.0 and zeros[0, 1] == 0
    assert zeros[0, 0] == 0
    wd = oracle.dequant_int4(codes, scales, zeros, k)
    assert wd[0, 5] == 15 * 0.06671142578125 == 1.00067138671875
    assert np.count_nonzero(wd) == 1
    # nibble order: element 2j in the low nibble of byte j
    assert codes[0, 2] == 0xF0
    w2 = np.zeros((1, 128), np.float16)
    w2[0, 4] = 1.0
    c2, _, _ = oracle.quantize_int4_g128(w2)
    assert c2[0, 2] == 0x0F


def test_int4_values_on_grid_round_trip_exactly():
    s = 2.0 ** -6
    for z in range(16):
        q = RNG.integers(0, 16, 128)
        q[0], q[1] = 0, 15                           # span the full code range
        w = ((q - z) * s).astype(np.float16)[None, :]
        codes, scales, zeros = oracle.quantize_int4_g128(w)
        assert scales.view(np.float16)[0, 0] == s
        wd = oracle.dequant_int4(codes, scales, zeros, 128)
        assert np.array_equal(wd[0], w[0].astype(np.float64))


def test_int4_nonfinite_and_shape_errors():
    w = np.zeros((2, 128), np.float16)
    w[1, 3] = np.inf
    with pytest.raises(oracle.OracleError) as e:
        oracle.quantize_int4_g128(w)
    assert e.value.status == oracle.ERR_NONFINITE
    with pytest.raises(oracle.OracleError) as e:
        oracle.quantize_int4_g128(np.zeros((1, 100), np.float16))
    assert e.value.status == oracle.ERR_SHAPE


def test_int4_deterministic():
    w = _groups_under_test()
    a = oracle.quantize_int4_g128(w)
    b = oracle.quantize_int4_g128(w.copy())
    for x, y in zip(a, b):
        assert np.array_equal(x, y)


# ------------------------------------------------------------------- FP8 ----
def _e4m3_table():
    return torch.arange(256, dtype=torch.int32).to(torch.uint8).view(torch.float8_e4m3fn).to(torch.float64).numpy()


def test_fp8_decode_all_codes_match_torch():
    ref = _e4m3_table()
    got = np.array([oracle.fp8_decode(c) for c in range(256)])
    nan = np.isnan(ref)
    assert list(np.nonzero(nan)[0]) == [0x7F, 0xFF]
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], ref[~nan])
    assert got[0x7E] == 448.0 and got[0x01] == 2.0 ** -9 and got[0x80] == 0.0 and np.signbit(got[0x80])


def _brute_force_e4m3(v: float) -> int:
    """Nearest finite E4M3 value to v, ties to the even code, saturating."""
    table = _e4m3_table()
    sign = 0x80 if np.signbit(v) else 0
    a = min(abs(v), 448.0)
    pos = table[:0x7F]                               # codes 0x00..0x7E, ascending
    d = np.abs(pos - a)
    best = np.nonzero(d == d.min())[0]
    code = int(best[0]) if len(best) == 1 else int([c for c in best if c % 2 == 0][0])
    return sign | code


def test_fp8_encode_all_fp16_inputs_match_torch_and_brute_force():
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    vals = bits.view(np.float16).astype(np.float64)
    finite = np.isfinite(vals)
    vals = vals[finite]
    got = np.array([oracle.fp8_encode(v) for v in vals], np.uint8)
    ref = torch.from_numpy(vals.astype(np.float32)).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    in_range = np.abs(vals) <= 448.0
    assert np.array_equal(got[in_range], ref[in_range])
    # saturation above 448 (torch produces NaN there instead)
    assert np.all((got[~in_range] & 0x7F) == 0x7E)
    # brute-force nearest at inputs that are not fp16 values (w / s at several scales)
    for s in (1.0, 2.0 ** -7, float(np.float32(0.05 / 448.0)), float(np.float32(1.7 / 448.0))):
        sample = RNG.normal(0, 0.02, 4000).astype(np.float16).astype(np.float64)
        for v in sample:
            assert oracle.fp8_encode(v / s) == _brute_force_e4m3(v / s), (v, s)


def test_fp8_quantize_scale_and_round_trip():
    w = np.stack([RNG.normal(0, 0.02, 512), RNG.normal(0, 1, 512), np.zeros(512),
                  RNG.normal(0, 1e-6, 512)]).astype(np.float16)
    w[0, 7] = np.float16(-0.0)
    codes, scales = oracle.quantize_fp8_e4m3(w)
    w64 = w.astype(np.float64)
    amax = np.abs(w64).max(axis=1)
    for r in range(w.shape[0]):
        exp = np.float32(1.0) if amax[r] == 0 else np.float32(amax[r] / 448.0)
        assert scales[r] == exp
    wd = oracle.dequant_fp8(codes, scales)
    table = _e4m3_table()
    for r in range(w.shape[0]):
        v = w64[r] / float(scales[r])
        # half the local E4M3 spacing: 2^(e-3)/2 for normals, 2^-10 for subnormals
        e = np.floor(np.log2(np.maximum(np.abs(v), 2.0 ** -6)))
        half = np.where(np.abs(v) < 2.0 ** -6, 2.0 ** -10, 2.0 ** (e - 4))
        assert np.all(np.abs(v - table[codes[r]]) <= half + 1e-300)
        assert np.all(np.abs(wd[r] - table[codes[r]] * float(scales[r])) == 0)
    assert codes[0, 7] == 0x80                     # -0 keeps its sign
    assert np.all(codes[2] == 0) and scales[2] == 1.0


def test_fp8_nonfinite_error():
    w = np.zeros((1, 32), np.float16)
    w[0, 0] = np.nan
    with pytest.raises(oracle.OracleError) as e:
        oracle.quantize_fp8_e4m3(w)
    assert e.value.status == oracle.ERR_NONFINITE
