"""Pins of the oracle's gating step against brute force, a hand-derived
worked example and invariants that follow from the definition."""
import json
import math
import os

import numpy as np
import pytest

import oracle


def brute_route(logits, k, local_begin, E_local):
    """Pure-Python: full softmax over all experts, a full sort by (logit desc,
    index asc), keep k, renormalise the kept probabilities."""
    T, E = len(logits), len(logits[0])
    ids, ws = [], []
    for t in range(T):
        row = [float(v) for v in logits[t]]
        mx = max(row)
        p = [math.exp(v - mx) for v in row]
        z = sum(p)
        p = [v / z for v in p]
        order = sorted(range(E), key=lambda i: (-row[i], i))[:k]
        s = sum(p[i] for i in order)
        ids.append([i - local_begin if 0 <= i - local_begin < E_local else -1 for i in order])
        ws.append([p[i] / s for i in order])
    return np.array(ids, dtype=np.int32), np.array(ws)


def test_worked_example(golden_dir):
    g = json.load(open(os.path.join(golden_dir, "route_worked.json")))
    L = np.array(g["logits"], dtype=np.float32)
    ids, w = oracle.route(L, g["top_k"], g["local_begin"], g["E_local"])
    np.testing.assert_array_equal(ids, np.array(g["local_ids"]))
    np.testing.assert_allclose(w, np.array(g["weights"]), rtol=0, atol=g["weights_tol"])
    gids, _ = oracle.route(L, g["top_k"], 0, L.shape[1])
    np.testing.assert_array_equal(gids, np.array(g["global_ids"]))


@pytest.mark.parametrize("E,k", [(4, 1), (4, 4), (8, 2), (8, 3), (16, 8), (16, 16)])
@pytest.mark.parametrize("kind", ["normal", "ties"])
def test_brute_force(E, k, kind):
    rng = np.random.default_rng(E * 100 + k)
    if kind == "normal":
        L = rng.standard_normal((40, E)).astype(np.float32)
    else:  # many exact ties, including signed zeros
        L = rng.choice(np.array([-1.0, -0.0, 0.0, 0.5, 2.0], dtype=np.float32), size=(40, E))
    for lb, El in [(0, E), (1, max(1, E // 2)), (E - 1, 1)]:
        ids, w = oracle.route(L, k, lb, El)
        bids, bw = brute_route(L.tolist(), k, lb, El)
        np.testing.assert_array_equal(ids, bids)
        np.testing.assert_allclose(w, bw, rtol=1e-12, atol=1e-15)


def test_invariants():
    rng = np.random.default_rng(5)
    L = (rng.standard_normal((200, 32)) * 4).astype(np.float32)
    for k in (1, 2, 8, 32):
        ids, w = oracle.route(L, k, 0, 32)
        np.testing.assert_allclose(w.sum(axis=1), 1.0, rtol=0, atol=1e-12)
        assert np.all(np.diff(w, axis=1) <= 1e-15), "weights follow descending logits"
        assert np.all(ids >= 0)
        for t in range(L.shape[0]):
            assert len(set(ids[t].tolist())) == k
        if k == 1:
            assert np.all(w == 1.0)
        if k == 32:  # all experts: the weights are the full softmax in slot order
            full = np.exp(L.astype(np.float64) - L.max(axis=1, keepdims=True))
            full /= full.sum(axis=1, keepdims=True)
            np.testing.assert_allclose(w, np.take_along_axis(full, ids, axis=1), rtol=1e-12)


def test_shift_invariance():
    """softmax weights do not change when a constant is added to a row."""
    rng = np.random.default_rng(6)
    L = rng.standard_normal((64, 16)).astype(np.float32)
    ids0, w0 = oracle.route(L, 4, 0, 16)
    ids1, w1 = oracle.route(L + np.float32(8.0), 4, 0, 16)
    np.testing.assert_array_equal(ids0, ids1)
    np.testing.assert_allclose(w0, w1, rtol=1e-5)


def test_rejects_bad_input():
    with pytest.raises(ValueError):
        oracle.route(np.zeros((2, 4), np.float32), 5, 0, 4)
    with pytest.raises(ValueError):
        oracle.route(np.array([[0.0, np.nan]], np.float32), 1, 0, 2)
