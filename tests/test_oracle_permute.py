"""Pins of the oracle's permutation step: brute force, a hand-derived worked
example and the round-trip invariants."""
import json
import os

import numpy as np
import pytest

import oracle


def brute_permute(ids, E_local, align):
    T, k = ids.shape
    flat = ids.reshape(-1).tolist()
    counts, offsets, r2a = [], [0], []
    a2r = [-1] * (T * k)
    for e in range(E_local):
        mine = [a for a in range(T * k) if flat[a] == e]
        counts.append(len(mine))
        size = ((len(mine) + align - 1) // align) * align
        for i, a in enumerate(mine):
            a2r[a] = offsets[-1] + i
        r2a.extend(mine + [-1] * (size - len(mine)))
        offsets.append(offsets[-1] + size)
    return counts, offsets, r2a, a2r


def test_worked_example(golden_dir):
    g = json.load(open(os.path.join(golden_dir, "permute_worked.json")))
    ids = np.array(g["ids"], dtype=np.int32)
    x = np.array(g["x"], dtype=np.uint16)
    p = oracle.permute(ids, g["E_local"], g["row_align"], x)
    np.testing.assert_array_equal(p.counts, g["counts"])
    np.testing.assert_array_equal(p.offsets, g["offsets"])
    np.testing.assert_array_equal(p.row_to_assign, g["row_to_assign"])
    np.testing.assert_array_equal(p.assign_to_row, g["assign_to_row"])
    np.testing.assert_array_equal(p.x_perm, np.array(g["x_perm"], dtype=np.uint16))


@pytest.mark.parametrize("T,k,E,align,p_local", [(1, 1, 1, 1, 1.0), (37, 2, 8, 16, 0.8), (64, 8, 32, 32, 0.3),
                                                  (200, 4, 5, 7, 1.0), (50, 3, 4, 1, 0.0)])
def test_brute_force(T, k, E, align, p_local):
    rng = np.random.default_rng(T + k + E)
    ids = rng.integers(0, E, size=(T, k)).astype(np.int32)
    ids[rng.random((T, k)) >= p_local] = -1
    p = oracle.permute(ids, E, align)
    c, o, r2a, a2r = brute_permute(ids, E, align)
    np.testing.assert_array_equal(p.counts, c)
    np.testing.assert_array_equal(p.offsets, o)
    np.testing.assert_array_equal(p.row_to_assign, r2a)
    np.testing.assert_array_equal(p.assign_to_row, a2r)


def test_round_trip_and_layout():
    rng = np.random.default_rng(11)
    T, k, E, align, H = 300, 8, 16, 32, 24
    ids = rng.integers(-1, E, size=(T, k)).astype(np.int32)
    x = rng.integers(0, 65535, size=(T, H)).astype(np.uint16)
    cap = T * min(k, E) + E * (align - 1)
    p = oracle.permute(ids, E, align, x, capacity=cap)
    assert p.row_to_assign.shape == (cap,)
    assert int(p.counts.sum()) == int(np.count_nonzero(ids >= 0))
    assert np.all(p.offsets % align == 0)
    seg = np.diff(p.offsets)
    assert np.all(seg >= p.counts) and np.all(seg < p.counts + align)
    flat = ids.reshape(-1)
    for a in range(T * k):
        r = p.assign_to_row[a]
        if flat[a] < 0:
            assert r == -1
            continue
        assert p.row_to_assign[r] == a
        assert p.offsets[flat[a]] <= r < p.offsets[flat[a]] + p.counts[flat[a]]
        assert np.array_equal(p.x_perm[r], x[a // k])     # bitwise copy
    pad = p.row_to_assign < 0
    assert np.all(p.x_perm[pad] == 0)


def test_fp8_scales_follow_rows():
    rng = np.random.default_rng(12)
    ids = rng.integers(-1, 4, size=(20, 2)).astype(np.int32)
    x = rng.integers(0, 255, size=(20, 256)).astype(np.uint8)
    xs = rng.random((20, 2)).astype(np.float32)
    p = oracle.permute(ids, 4, 8, x, None, xs)
    for a, r in enumerate(p.assign_to_row):
        if r >= 0:
            assert np.array_equal(p.x_perm_scales[r], xs[a // 2])
    assert np.all(p.x_perm_scales[p.row_to_assign < 0] == 0)


def test_rejects_bad_ids():
    with pytest.raises(ValueError):
        oracle.permute(np.array([[0, 4]], np.int32), 4, 1)
    with pytest.raises(ValueError):
        oracle.permute(np.array([[0, -2]], np.int32), 4, 1)
    with pytest.raises(ValueError):
        oracle.permute(np.array([[0, 1]], np.int32), 4, 4, capacity=4)


# ----------------------------------------------------------------------------- masked layout

def brute_permute_masked(ids, E_local, slots):
    T, k = ids.shape
    flat = ids.reshape(-1).tolist()
    counts = [0] * E_local
    r2a = [-1] * (E_local * slots)
    a2r = [-1] * (T * k)
    for a in range(T * k):
        e = flat[a]
        if e < 0:
            continue
        row = e * slots + counts[e]
        counts[e] += 1
        r2a[row] = a
        a2r[a] = row
    return counts, [e * slots for e in range(E_local + 1)], r2a, a2r


def test_masked_worked_example(golden_dir):
    g = json.load(open(os.path.join(golden_dir, "permute_masked_worked.json")))
    ids = np.array(g["ids"], dtype=np.int32)
    x = np.array(g["x"], dtype=np.uint16)
    p = oracle.permute_masked(ids, g["E_local"], g["slots"], x)
    np.testing.assert_array_equal(p.counts, g["counts"])
    np.testing.assert_array_equal(p.offsets, g["offsets"])
    np.testing.assert_array_equal(p.row_to_assign, g["row_to_assign"])
    np.testing.assert_array_equal(p.assign_to_row, g["assign_to_row"])
    np.testing.assert_array_equal(p.x_perm, np.array(g["x_perm"], dtype=np.uint16))


@pytest.mark.parametrize("T,k,E,p_local", [(1, 1, 1, 1.0), (37, 2, 8, 0.8), (64, 8, 32, 0.3), (50, 3, 4, 0.0)])
def test_masked_brute_force(T, k, E, p_local):
    rng = np.random.default_rng(T * 3 + k + E)
    ids = np.stack([rng.permutation(E)[:k] if k <= E else rng.integers(0, E, k) for _ in range(T)]).astype(np.int32)
    ids[rng.random((T, k)) >= p_local] = -1
    slots = (T + 31) // 32 * 32
    p = oracle.permute_masked(ids, E, slots)
    c, o, r2a, a2r = brute_permute_masked(ids, E, slots)
    np.testing.assert_array_equal(p.counts, c)
    np.testing.assert_array_equal(p.offsets, o)
    np.testing.assert_array_equal(p.row_to_assign, r2a)
    np.testing.assert_array_equal(p.assign_to_row, a2r)


def test_masked_round_trip_and_regions():
    """Every local slot has its own row inside its expert's region, in
    ascending assignment order, and the gathered row is a bitwise copy of the
    token's activations; rows past a region's count are -1 / zero."""
    rng = np.random.default_rng(13)
    T, k, E, H = 200, 4, 12, 16
    ids = np.stack([rng.permutation(E)[:k] for _ in range(T)]).astype(np.int32)
    ids[rng.random((T, k)) < 0.3] = -1
    x = rng.integers(0, 65535, size=(T, H)).astype(np.uint16)
    slots = 224
    p = oracle.permute_masked(ids, E, slots, x)
    flat = ids.reshape(-1)
    assert int(p.counts.sum()) == int(np.count_nonzero(flat >= 0))
    for e in range(E):
        region = p.row_to_assign[e * slots:(e + 1) * slots]
        mine = region[:p.counts[e]]
        assert np.all(np.diff(mine) > 0)                    # ascending a
        assert np.all(flat[mine] == e)
        assert np.all(region[p.counts[e]:] == -1)
    for a in range(T * k):
        r = p.assign_to_row[a]
        if flat[a] < 0:
            assert r == -1
            continue
        assert p.row_to_assign[r] == a
        assert np.array_equal(p.x_perm[r], x[a // k])
    assert np.all(p.x_perm[p.row_to_assign < 0] == 0)


def test_masked_rejects_small_regions():
    with pytest.raises(ValueError):
        oracle.permute_masked(np.array([[0, 1], [0, 2]], np.int32), 3, 1)
