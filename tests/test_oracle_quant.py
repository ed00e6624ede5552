"""Pins of the oracle's fp8 intermediate quantization (reading taken for the
fp8 path: h is stored per row and 128 columns with scale = max(amax, 1e-4) /
448, as OCP E4M3FN codes rounded to nearest even and saturating at +-448).
The encoder is checked against the decoder (itself pinned to the format's
definition), against values derived by hand from the format, and the row
quantizer against its closed forms."""
import numpy as np

import oracle


def _finite_codes():
    c = np.arange(256, dtype=np.uint8)
    return c[~np.isnan(oracle.e4m3_to_f64(c))]


def test_e4m3_round_trip_every_finite_code():
    c = _finite_codes()
    assert len(c) == 254                                     # 0x7F and 0xFF are NaN
    np.testing.assert_array_equal(oracle.e4m3_quantize(oracle.e4m3_to_f64(c)), c)


def test_e4m3_midpoints_round_to_even_and_neighbours_to_nearest():
    v = oracle.e4m3_to_f64(np.arange(0x7F, dtype=np.uint8))  # 0x00..0x7E ascending
    lo, hi = np.arange(0x7E), np.arange(1, 0x7F)
    mid = (v[:-1] + v[1:]) / 2
    want = np.where(lo % 2 == 0, lo, hi)
    np.testing.assert_array_equal(oracle.e4m3_quantize(mid), want)
    np.testing.assert_array_equal(oracle.e4m3_quantize(-mid), want | 0x80)
    eps = (v[1:] - v[:-1]) * 1e-3
    np.testing.assert_array_equal(oracle.e4m3_quantize(mid - eps), lo)
    np.testing.assert_array_equal(oracle.e4m3_quantize(mid + eps), hi)


def test_e4m3_hand_derived_values():
    # 0.1 = 2^-4 * 1.6 -> mantissa 4.8/8 rounds to 5/8: 0.1015625, exponent field 3 -> 0b0_0011_101
    # 3.14 = 2^1 * 1.57 -> 4.56/8 rounds to 5/8: 3.25, exponent field 8 -> 0b0_1000_101
    # 300 lies between 288 (2^8 * 9/8) and 320 (2^8 * 10/8), nearer 288 -> 0b1_1111_001 for -300
    # 2^-10 is half the smallest subnormal 2^-9: a tie, to the even code 0; 0.001 is nearer 2^-9
    x = np.array([0.1, 3.14, -300.0, 448.0, 500.0, -1e6, 2.0 ** -10, 0.001, -0.0])
    want = np.array([0x1D, 0x45, 0xF9, 0x7E, 0x7E, 0xFE, 0x00, 0x01, 0x80], dtype=np.uint8)
    np.testing.assert_array_equal(oracle.e4m3_quantize(x), want)


def test_quantize_rows_closed_forms():
    rng = np.random.default_rng(3)
    h = rng.standard_normal((5, 384))
    h[2, 128:256] = 0.0                                      # an all-zero group
    codes, sc = oracle.quantize_rows(h)
    g = h.reshape(5, 3, 128)
    amax = np.abs(g).max(axis=2)
    np.testing.assert_allclose(sc[amax > 0], amax[amax > 0] / 448.0, rtol=0, atol=0)
    assert sc[2, 1] == 1e-4 / 448.0 and np.all(codes[2, 128:256] == 0)
    # the element of largest magnitude in each group is coded exactly as +-448
    arg = np.abs(g).argmax(axis=2)
    top = np.take_along_axis(codes.reshape(5, 3, 128), arg[:, :, None], axis=2)[:, :, 0]
    top_sign = np.take_along_axis(g, arg[:, :, None], axis=2)[:, :, 0] < 0
    ok = amax > 0
    np.testing.assert_array_equal(top[ok], np.where(top_sign, 0xFE, 0x7E)[ok])
    # codes do not depend on a positive common factor (while every amax stays above the floor)
    codes2, sc2 = oracle.quantize_rows(h * 8.0)
    np.testing.assert_array_equal(codes2, codes)
    np.testing.assert_allclose(sc2[ok], 8.0 * sc[ok], rtol=1e-15)


def test_h_fp8_option_closed_form():
    """x = e0; gate column 10 for both outputs, up column (1, 0.3): h = silu(10) * (1, 0.3).
    In fp8, 0.3 of the group maximum is 134.4 on the 448 scale, which rounds to
    128 (the neighbours are 128 and 144): the second output becomes 2/7 of the
    first.  Down projection: identity on the two channels."""
    H = I = 128
    x = np.zeros((1, H)); x[0, 0] = 1.0
    wg = np.zeros((I, H)); wg[:2, 0] = 10.0
    wu = np.zeros((I, H)); wu[0, 0] = 1.0; wu[1, 0] = 0.3
    wd = np.eye(H, I)
    s10 = 10.0 / (1.0 + np.exp(-10.0))
    plain = oracle.expert_ffn(x, wg, wu, wd)[0]
    quant = oracle.expert_ffn(x, wg, wu, wd, h_fp8=True)[0]
    np.testing.assert_allclose(plain[:2], [s10, 0.3 * s10], rtol=1e-15)
    np.testing.assert_allclose(quant[:2], [s10, s10 * 2.0 / 7.0], rtol=1e-15)
    assert np.all(quant[2:] == 0.0)
