"""The seeded generator: determinism, storage-format rounding against brute
force, and the workload shapes it is meant to produce."""
import numpy as np
import pytest

import oracle
from workload import CONFIGS, bf16_bits, custom_config, e4m3_codes, make_layer, make_phase
from workload.gen import zipf_bias


def _nearest_even(values, grid_vals, grid_codes):
    """Brute force: nearest representable value, ties to the even code."""
    out = []
    for v in values:
        d = np.abs(grid_vals - v)
        best = np.nonzero(d == d.min())[0]
        cs = grid_codes[best]
        even = cs[cs % 2 == 0]
        out.append(int(even[0] if len(even) else cs[0]))
    return np.array(out)


def test_bf16_rounding_brute_force():
    rng = np.random.default_rng(1)
    v = (rng.standard_normal(400) * 10 ** rng.uniform(-3, 3, 400)).astype(np.float32)
    ties = np.array([1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -(2.0 + 2 ** -7), 3.0 + 2 ** -7], np.float32)
    v = np.concatenate([v, ties])
    got = bf16_bits(v)
    for x, b in zip(v, got):
        hi = np.uint32(np.float32(x).view(np.uint32)) >> 16
        cands = np.array([hi, hi + 1], dtype=np.uint32)
        vals = (cands << 16).view(np.float32).astype(np.float64)
        d = np.abs(vals - float(x))
        if d[0] < d[1] or (d[0] == d[1] and cands[0] % 2 == 0):
            want = cands[0]
        else:
            want = cands[1]
        assert int(b) == int(want), (x, hex(b), hex(want))
    assert list(bf16_bits(ties)) == [0x3F80, 0x3F82, 0xC000, 0x4040]


def test_e4m3_encoding_brute_force():
    codes = np.arange(0, 127)
    vals = oracle.e4m3_to_f64(codes.astype(np.uint8))
    rng = np.random.default_rng(2)
    v = np.concatenate([vals, 0.5 * (vals[1:] + vals[:-1]), rng.uniform(0, 448, 3000),
                        rng.uniform(0, 2 ** -6, 500), [448.0, 450.0, 463.9, 464.0, 1e4]]).astype(np.float32)
    for sign in (1.0, -1.0):
        got = e4m3_codes(np.float32(sign) * v)
        want = _nearest_even(np.minimum(v.astype(np.float64), 448.0), vals, codes)
        if sign < 0:
            want = np.where(want == 0, 0, want) | 0x80
            want[v == 0] = 0x80
        np.testing.assert_array_equal(got, want.astype(np.uint8))


def test_determinism_and_independence():
    cfg = custom_config(2, cfg_id=101, H=128, I=64, E_global=32, E_local=8, decode_tokens=16)
    a = make_layer(cfg, 0)
    b = make_layer(cfg, 0)
    c = make_layer(cfg, 1) if cfg.n_layers > 1 else make_layer(custom_config(2, cfg_id=101, H=128, I=64,
                                                                             E_global=32, E_local=8,
                                                                             decode_tokens=16, n_layers=2,
                                                                             zipf_s=(1.1, 1.1)), 1)
    for k in ("w_gate_up", "w_down"):
        np.testing.assert_array_equal(a.weights[k], b.weights[k])
        assert not np.array_equal(a.weights[k], c.weights[k])
    np.testing.assert_array_equal(a.phases[0].logits, b.phases[0].logits)
    np.testing.assert_array_equal(a.phases[0].x, b.phases[0].x)


def test_zipf_bias_hot_expert_is_local_zero():
    cfg = CONFIGS[2]
    b = zipf_bias(cfg, 0)
    assert b[cfg.local_begin] == np.float32(1.0)
    ranks_back = np.sort(b)[::-1]
    np.testing.assert_allclose(ranks_back, np.arange(1, 257, dtype=np.float64) ** -1.1, rtol=1e-6)


def test_fp8_inputs_scale_rule():
    cfg = custom_config(5, cfg_id=105, H=256, I=128, E_global=16, E_local=2, prefill_tokens=8, decode_tokens=0)
    lay = make_layer(cfg, 0, keep_f32=True)
    w, s, f = lay.weights["w_gate_up"][0], lay.weights["w_gate_up_scales"][0], lay.weights["w_gate_up_f32"][0]
    amax = np.abs(f.reshape(2, 128, 2, 128)).max(axis=(1, 3))
    np.testing.assert_allclose(s, np.maximum(amax, 1e-4) / 448.0, rtol=1e-7)
    deq = oracle.dequant_weight(w, s)
    assert np.max(np.abs(deq - f)) <= np.max(s) * 448 * 2 ** -4 + 1e-12     # half an e4m3 ulp at most
    ph = lay.phases[0]
    assert ph.x.dtype == np.uint8 and ph.x_scales.shape == (8, 2)


@pytest.mark.slow
def test_decode_workload_shape():
    """Config 2's routing lands a few hundred local rows with a hot expert."""
    cfg = CONFIGS[2]
    ph = make_phase(cfg, 0, "decode")
    ids, _ = oracle.route(ph.logits, cfg.top_k, cfg.local_begin, cfg.E_local)
    counts = np.bincount(ids[ids >= 0], minlength=cfg.E_local)
    assert 450 <= counts.sum() <= 800
    assert counts.argmax() == 0 and counts.min() > 0
