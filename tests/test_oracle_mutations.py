"""Mutation check of the oracle's pins.

Each mutant plants one plausible mistake in a copy of the oracle's source (a
dropped term, a wrong sign or index, a transposed operand), loads the copy as
a module, points the `oracle` package at it and runs the pin tests.  At least
one pin must fail for every mutant; the real oracle must pass them all.
"""
import importlib.util
import os
import sys
import types

import pytest

import oracle
import oracle.moe as real

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = open(real.__file__).read()


def _load(path, name):
    spec = importlib.util.spec_from_file_location(name, path)
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


PINS = {n: _load(os.path.join(HERE, f"test_oracle_{n}.py"), f"_pins_{n}")
        for n in ("route", "permute", "ffn", "policy", "quant")}
GOLDEN = os.path.join(HERE, "golden")


def _run_pins():
    r, p, f, q, z = PINS["route"], PINS["permute"], PINS["ffn"], PINS["policy"], PINS["quant"]
    calls = [
        lambda: r.test_worked_example(GOLDEN), lambda: r.test_brute_force(8, 3, "ties"),
        lambda: r.test_brute_force(16, 8, "normal"), r.test_invariants,
        lambda: p.test_worked_example(GOLDEN), lambda: p.test_brute_force(37, 2, 8, 16, 0.8),
        p.test_round_trip_and_layout, p.test_fp8_scales_follow_rows,
        lambda: p.test_masked_worked_example(GOLDEN), lambda: p.test_masked_brute_force(37, 2, 8, 0.8),
        p.test_masked_round_trip_and_regions,
        lambda: f.test_basis_closed_form(GOLDEN), lambda: f.test_formats(GOLDEN), f.test_block_dequant,
        f.test_dense_gate_matrix_form, f.test_identical_experts_reduce_to_dense_ffn, f.test_combine_properties,
        f.test_permute_combine_round_trip_is_identity, f.test_fp8_path_dequantizes_same_codes,
        q.test_x_moe_eq3, q.test_quota_eq4,
        z.test_e4m3_round_trip_every_finite_code, z.test_e4m3_midpoints_round_to_even_and_neighbours_to_nearest,
        z.test_e4m3_hand_derived_values, z.test_quantize_rows_closed_forms, z.test_h_fp8_option_closed_form,
    ]
    failed = 0
    for c in calls:
        try:
            c()
        except Exception:  # an assertion or an error raised by the mutant both count
            failed += 1
    return failed


MUTANTS = [
    ("route: ascending order", "np.lexsort((index, -L), axis=-1)", "np.lexsort((index, L), axis=-1)"),
    ("route: ties to the higher index", "np.lexsort((index, -L), axis=-1)", "np.lexsort((-index, -L), axis=-1)"),
    ("route: softmax not renormalised", "w = ex / ex.sum(axis=1, keepdims=True)",
     "w = ex / np.exp(L - m).sum(axis=1, keepdims=True)"),
    ("route: local id off by one", "local = sel - local_begin", "local = sel - local_begin + 1"),
    ("route: local range too wide", "(local < E_local)", "(local <= E_local)"),
    ("permute: padding ignored", "-(-counts[e] // row_align) * row_align", "counts[e]"),
    ("permute: rows in descending order", 'kind="stable")]', 'kind="stable")][::-1]'),
    ("permute: wrong source token", "x[row_to_assign[valid] // k]", "x[row_to_assign[valid] % k]"),
    ("masked: region start off by one", "offsets = np.arange(E_local + 1, dtype=np.int64) * slots",
     "offsets = np.arange(E_local + 1, dtype=np.int64) * slots + 1"),
    ("masked: rows in descending order", "for a in range(T * k):                          # ascending a",
     "for a in reversed(range(T * k)):                # ascending a"),
    ("masked: wrong source token", "xp[valid] = x[row_to_assign[valid] // k]\n        res.x_perm = xp\n        if x_scales is not None:\n            xs = np.zeros((cap,) + x_scales.shape[1:], dtype=x_scales.dtype)\n            xs[valid] = x_scales[row_to_assign[valid] // k]\n            res.x_perm_scales = xs\n    return res\n\n\n# -----",
     "xp[valid] = x[row_to_assign[valid] % k]\n        res.x_perm = xp\n        if x_scales is not None:\n            xs = np.zeros((cap,) + x_scales.shape[1:], dtype=x_scales.dtype)\n            xs[valid] = x_scales[row_to_assign[valid] // k]\n            res.x_perm_scales = xs\n    return res\n\n\n# -----"),
    ("ffn: up used as gate", "g = x_rows @ w_gate.T", "g = x_rows @ w_up.T"),
    ("ffn: sigmoid instead of silu", "h = g / (1.0 + np.exp(-g)) * u", "h = 1.0 / (1.0 + np.exp(-g)) * u"),
    ("ffn: gate/up halves swapped", "return gu[:I], gu[I:], wd", "return gu[I:], gu[:I], wd"),
    ("ffn: down not transposed", "return h @ w_down.T", "return h @ w_down.T[::-1]"),
    ("combine: weight dropped", "y[hit] += w[hit, j][:, None] * y_perm[r[hit]]", "y[hit] += y_perm[r[hit]]"),
    ("combine: slot weight misindexed", "y[hit] += w[hit, j]", "y[hit] += w[hit, 0]"),
    ("dequant: block scales transposed", "s[:, None, :, None]", "s.T[:, None, :, None]"),
    ("dequant: row scales reversed", "[:, :, None]).reshape(T, H)", "[:, ::-1, None]).reshape(T, H)"),
    ("e4m3: exponent bias", "2.0 ** (e - 7)", "2.0 ** (e - 8)"),
    ("e4m3: subnormal scale", "(m / 8.0) * 2.0 ** -6", "(m / 8.0) * 2.0 ** -7"),
    ("bf16: wrong shift", "astype(np.uint32) << 16", "astype(np.uint32) << 15"),
    ("x_moe: floor instead of ceil", "-(-int(m) // M_t)", "(int(m) // M_t)"),
    ("quota: Q_max cap dropped", "return min(int(q_max), rounded)", "return rounded"),
    ("quota: ratio inverted", "num, den = int(q) * int(x_moe_now), int(x_moe_star)",
     "num, den = int(q) * int(x_moe_star), max(1, int(x_moe_now))"),
    ("e4m3 encode: ties to the odd code", "(d_lo == d_hi) & (lo % 2 == 0)", "(d_lo == d_hi) & (lo % 2 == 1)"),
    ("e4m3 encode: saturates at 240", "np.minimum(np.abs(v), 448.0)", "np.minimum(np.abs(v), 240.0)"),
    ("h quant: scale floor dropped", "np.maximum(np.abs(g).max(axis=2), floor)", "np.abs(g).max(axis=2)"),
    ("h quant: wrong full-scale code", "floor) / qmax", "floor) / (qmax / 2)"),
    ("h quant: option ignored", "    if h_fp8:\n        codes, sc", "    if False:\n        codes, sc"),
    ("quota: no rounding to the multiple", "rounded = c * (-(-num // (den * c)))", "rounded = -(-num // den)"),
]


def _patched(monkeypatch, mod):
    for name in dir(real):
        if not name.startswith("__") and hasattr(mod, name):
            monkeypatch.setattr(real, name, getattr(mod, name), raising=False)
            if hasattr(oracle, name):
                monkeypatch.setattr(oracle, name, getattr(mod, name))


def test_real_oracle_passes_all_pins():
    assert _run_pins() == 0


@pytest.mark.parametrize("label,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_mutant_is_caught(monkeypatch, label, old, new):
    assert SRC.count(old) >= 1, f"mutation site vanished: {old!r}"
    mod = types.ModuleType("oracle_mutant")
    monkeypatch.setitem(sys.modules, "oracle_mutant", mod)
    exec(compile(SRC.replace(old, new), "oracle_mutant", "exec"), mod.__dict__)
    _patched(monkeypatch, mod)
    assert _run_pins() > 0, f"no pin caught mutant: {label}"


def test_unmutated_copy_passes_all_pins(monkeypatch):
    """Control: loading the unchanged source the same way breaks nothing."""
    mod = types.ModuleType("oracle_mutant")
    monkeypatch.setitem(sys.modules, "oracle_mutant", mod)
    exec(compile(SRC, "oracle_mutant", "exec"), mod.__dict__)
    _patched(monkeypatch, mod)
    assert _run_pins() == 0
