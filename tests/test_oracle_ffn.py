"""Pins of the oracle's expert FFN, combine and storage-format decoding."""
import json
import os

import numpy as np
import pytest

import oracle
from workload import bf16_bits


def _weights_bf16(rng, E, H, I, std=0.05):
    return dict(w_gate_up=bf16_bits(rng.standard_normal((E, 2 * I, H)).astype(np.float32) * std),
                w_down=bf16_bits(rng.standard_normal((E, H, I)).astype(np.float32) * std))


def test_basis_closed_form(golden_dir):
    g = json.load(open(os.path.join(golden_dir, "ffn_basis.json")))
    out = oracle.expert_ffn(np.array([g["x"]]), np.array(g["w_gate"]), np.array(g["w_up"]), np.array(g["w_down"]))
    np.testing.assert_allclose(out[0], g["out"], rtol=0, atol=g["tol"])


def test_formats(golden_dir):
    g = json.load(open(os.path.join(golden_dir, "formats.json")))
    for h, v in g["bf16"]:
        got = oracle.bf16_to_f64(np.array([int(h, 16)], np.uint16))[0]
        assert got == v and np.signbit(got) == np.signbit(v)
    for h, v in g["e4m3"]:
        assert oracle.e4m3_to_f64(np.array([int(h, 16)], np.uint8))[0] == v
    for h in g["e4m3_nan"]:
        assert np.isnan(oracle.e4m3_to_f64(np.array([int(h, 16)], np.uint8))[0])
    # every finite code, by sign symmetry and monotonicity of the positive half
    pos = oracle.e4m3_to_f64(np.arange(0, 127, dtype=np.uint8))
    assert np.all(np.diff(pos) > 0)
    np.testing.assert_array_equal(oracle.e4m3_to_f64(np.arange(128, 255, dtype=np.uint8)), -pos)


def test_block_dequant():
    codes = np.full((256, 384), 0x38, np.uint8)            # every code is 1.0
    scales = np.array([[2.0, 3.0, 5.0], [7.0, 11.0, 13.0]], np.float32)
    w = oracle.dequant_weight(codes, scales)
    for bi in range(2):
        for bj in range(3):
            assert np.all(w[bi * 128:(bi + 1) * 128, bj * 128:(bj + 1) * 128] == scales[bi, bj])
    rows = oracle.dequant_rows(np.full((2, 256), 0xB8, np.uint8), np.array([[2, 4], [8, 16]], np.float32))
    np.testing.assert_array_equal(rows[0, :128], -2.0)
    np.testing.assert_array_equal(rows[1, 128:], -16.0)


def test_dense_gate_matrix_form():
    """y = sum_e G[t,e] FFN_e(x_t) with the sparse gate matrix G, every expert
    evaluated densely on every token (einsum), against the gathered oracle."""
    rng = np.random.default_rng(21)
    T, Eg, El, lb, k, H, I = 40, 12, 5, 3, 3, 16, 8
    L = rng.standard_normal((T, Eg)).astype(np.float32)
    x = bf16_bits(rng.standard_normal((T, H)).astype(np.float32))
    W = _weights_bf16(rng, El, H, I)
    res = oracle.moe_local_share(L, x, W, k, lb, El, row_align=4)
    xf = oracle.bf16_to_f64(x)
    gu = oracle.bf16_to_f64(W["w_gate_up"])
    wd = oracle.bf16_to_f64(W["w_down"])
    g = np.einsum("th,eih->tei", xf, gu[:, :I])
    u = np.einsum("th,eih->tei", xf, gu[:, I:])
    h = g * (1.0 / (1.0 + np.exp(-g))) * u
    out = np.einsum("tei,ehi->teh", h, wd)
    G = np.zeros((T, El))
    ids, w = res["ids"], res["w"]
    for t in range(T):
        for j in range(k):
            if ids[t, j] >= 0:
                G[t, ids[t, j]] += w[t, j]
    y_dense = np.einsum("te,teh->th", G, out)
    np.testing.assert_allclose(res["y"], y_dense, rtol=1e-12, atol=1e-14)


def test_identical_experts_reduce_to_dense_ffn():
    rng = np.random.default_rng(22)
    T, E, k, H, I = 30, 8, 2, 16, 24
    L = rng.standard_normal((T, E)).astype(np.float32)
    x = bf16_bits(rng.standard_normal((T, H)).astype(np.float32))
    one = _weights_bf16(rng, 1, H, I)
    W = dict(w_gate_up=np.repeat(one["w_gate_up"], E, 0), w_down=np.repeat(one["w_down"], E, 0))
    res = oracle.moe_local_share(L, x, W, k, 0, E, row_align=8)
    gu = oracle.bf16_to_f64(one["w_gate_up"][0])
    dense = oracle.expert_ffn(oracle.bf16_to_f64(x), gu[:I], gu[I:], oracle.bf16_to_f64(one["w_down"][0]))
    np.testing.assert_allclose(res["y"], dense, rtol=1e-12, atol=1e-14)


def test_zero_gate_gives_zero():
    rng = np.random.default_rng(23)
    T, E, k, H, I = 20, 4, 2, 8, 8
    W = _weights_bf16(rng, E, H, I)
    W["w_gate_up"][:, :I] = 0
    res = oracle.moe_local_share(rng.standard_normal((T, E)).astype(np.float32),
                                 bf16_bits(rng.standard_normal((T, H)).astype(np.float32)), W, k, 0, E, 4)
    assert np.all(res["y"] == 0.0)


def test_combine_properties():
    rng = np.random.default_rng(24)
    T, Eg, El, k, H, I = 50, 16, 4, 4, 8, 8
    L = rng.standard_normal((T, Eg)).astype(np.float32)
    L[:5, :El] = -30.0                     # tokens 0..4 pick no local expert
    x = bf16_bits(rng.standard_normal((T, H)).astype(np.float32))
    W = _weights_bf16(rng, El, H, I)
    res = oracle.moe_local_share(L, x, W, k, 0, El, 4)
    assert np.all(res["ids"][:5] < 0)
    assert np.all(res["y"][:5] == 0.0)     # exactly zero, not merely small
    # linearity in the weights
    y2 = oracle.combine(res["y_perm"], res["perm"].assign_to_row, 2.5 * res["w"], T, k)
    np.testing.assert_allclose(y2, 2.5 * res["y"], rtol=1e-13, atol=1e-15)
    # token order does not matter: permuting tokens permutes outputs
    perm = rng.permutation(T)
    res_p = oracle.moe_local_share(L[perm], x[perm], W, k, 0, El, 4)
    np.testing.assert_allclose(res_p["y"], res["y"][perm], rtol=1e-12, atol=1e-14)


def test_permute_combine_round_trip_is_identity():
    """All experts local and weights summing to one: combining the gathered
    inputs themselves returns every token's input."""
    rng = np.random.default_rng(25)
    T, E, k, H = 64, 8, 3, 32
    L = rng.standard_normal((T, E)).astype(np.float32)
    x = bf16_bits(rng.standard_normal((T, H)).astype(np.float32))
    ids, w = oracle.route(L, k, 0, E)
    p = oracle.permute(ids, E, 16, x)
    y = oracle.combine(oracle.bf16_to_f64(p.x_perm), p.assign_to_row, w, T, k)
    np.testing.assert_allclose(y, oracle.bf16_to_f64(x), rtol=1e-14, atol=1e-14)


def test_token_output_matches_batched():
    rng = np.random.default_rng(26)
    T, Eg, El, k, H, I = 24, 16, 8, 4, 16, 16
    L = rng.standard_normal((T, Eg)).astype(np.float32)
    x = bf16_bits(rng.standard_normal((T, H)).astype(np.float32))
    W = _weights_bf16(rng, El, H, I)
    res = oracle.moe_local_share(L, x, W, k, 2, El, 8)
    cache = {}
    xf = oracle.bf16_to_f64(x)
    for t in range(T):
        yt = oracle.token_output(xf[t], res["ids"][t], res["w"][t], W, cache)
        np.testing.assert_allclose(yt, res["y"][t], rtol=1e-12, atol=1e-14)


def test_fp8_path_dequantizes_same_codes():
    """fp8 inputs: the oracle works on exactly the dequantized codes, so an
    all-0x38 (1.0) input with unit scales equals the bf16 path on ones."""
    T, E, k, H, I = 8, 2, 1, 128, 128
    L = np.tile(np.array([[1.0, 0.0]], np.float32), (T, 1))
    x8 = np.full((T, H), 0x38, np.uint8)
    xs = np.full((T, 1), 0.5, np.float32)
    W8 = dict(w_gate_up=np.full((E, 2 * I, H), 0x30, np.uint8),       # 0.5
              w_gate_up_scales=np.full((E, 2, 1), 0.25, np.float32),
              w_down=np.full((E, H, I), 0x38, np.uint8),
              w_down_scales=np.full((E, 1, 1), 0.125, np.float32))
    r8 = oracle.moe_local_share(L, x8, W8, k, 0, E, 4, x_scales=xs)
    g = H * 0.5 * (0.5 * 0.25)           # x = 0.5, w = 0.125 per element
    h = g / (1 + np.exp(-g)) * g
    y = I * h * 0.125
    np.testing.assert_allclose(r8["y"], np.full((T, H), y), rtol=1e-13)


def test_two_stage_split_composes_to_the_ffn():
    """grouped_down(grouped_hidden(x)) is grouped_ffn(x), segment by segment,
    with rows outside the segments zero in both stages."""
    rng = np.random.default_rng(21)
    E, H, I = 3, 64, 96
    counts = np.array([5, 0, 7])
    offsets = np.array([0, 8, 8, 16])
    x = rng.standard_normal((16, H))
    w = {"w_gate_up": bf16_bits((rng.standard_normal((E, 2 * I, H)) * 0.1).astype(np.float32)),
         "w_down": bf16_bits((rng.standard_normal((E, H, I)) * 0.1).astype(np.float32))}
    h = oracle.grouped_hidden(x, counts, offsets, w)
    y = oracle.grouped_down(h, counts, offsets, w)
    np.testing.assert_allclose(y, oracle.grouped_ffn(x, counts, offsets, w), rtol=1e-12, atol=1e-12)
    assert np.all(h[5:8] == 0) and np.all(y[5:8] == 0) and np.all(y[15:] == 0)
