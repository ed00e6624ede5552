"""CPU checks of the persistent scheduler's index arithmetic (row tiles of
Eq. (3), weight-sharing groups, per-XCD queues, tile numbering and the claim
resolution through a workgroup's LDS cache), through moe_sched_layout: the
host build of the very functions the kernel runs.  Ragged counts, empty
experts, one-tile and thousand-tile queues, every group size."""
import os

import numpy as np
import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB = os.path.join(ROOT, "paper_2607_18002_amd", "libmoe_apk.so")
pytestmark = pytest.mark.skipif(not os.path.exists(LIB), reason="library not built (run __graft_entry__.build())")


def _contiguous_offsets(counts, align=32):
    off = np.zeros(len(counts), np.int64)
    run = 0
    for e, c in enumerate(counts):
        off[e] = run
        run += -(-int(c) // align) * align
    return off


def _check(counts, offsets, M_t, gmax, n1, n2):
    from paper_2607_18002_amd import ops
    rt, gr, qu, tl = ops.moe_sched_layout(counts, offsets, M_t, gmax, n1, n2)
    x = oracle.x_moe(counts, M_t)
    assert len(rt) == x
    assert len(tl) == oracle.count_tiles(counts, M_t, n1, 1) + oracle.count_tiles(counts, M_t, n2, 1)
    # row tiles: one run per expert, near-equal heights in whole 32-row blocks,
    # partitioning the expert's rows from its segment start
    p = 0
    for e, c in enumerate(counts):
        nt = -(-int(c) // M_t) if c > 0 else 0
        mine = rt[p:p + nt]
        assert np.all(mine[:, 0] == e) and np.array_equal(mine[:, 1], np.arange(nt))
        if nt:
            assert int(mine[:, 2].sum()) == c
            assert np.all((mine[:, 2] >= 1) & (mine[:, 2] <= M_t))
            assert np.all(mine[:-1, 2] % 32 == 0)
            assert mine[:, 2].max() - mine[:, 2].min() <= 32
            assert np.array_equal(mine[:, 3], offsets[e] + np.concatenate([[0], np.cumsum(mine[:-1, 2])]))
        # groups: inside the expert, at most gmax row tiles, near-equal sizes
        if nt:
            g = gr[p:p + nt]
            assert np.all((g[:, 0] >= p) & (g[:, 0] + g[:, 1] <= p + nt))
            assert np.all((g[:, 0] <= np.arange(p, p + nt)) & (np.arange(p, p + nt) < g[:, 0] + g[:, 1]))
            sizes = [int(s) for f, s in {(int(a), int(b)) for a, b in g}]
            assert max(sizes) <= gmax and max(sizes) - min(sizes) <= 1
            assert sum(sizes) == nt
        p += nt
    # queues: contiguous ranges in order, cut only between groups, balanced to a group
    assert qu[0, 0] == 0 and int(qu[:, 1].sum()) == x
    assert np.array_equal(qu[1:, 0], qu[:-1, 0] + qu[:-1, 1])
    starts = {int(a) for a, _ in gr} | {x}
    for lo, n in qu:
        assert lo in starts or n == 0
    gsize = int(gr[:, 1].max()) if x else 0
    for q in range(8):
        assert abs(int(qu[q, 0]) - x * q // 8) <= gsize
        # exactly the group boundary nearest to q/8 of the row tiles, ties to the lower one
        assert int(qu[q, 0]) == min(sorted(starts), key=lambda b: (abs(b - x * q // 8), b))
    # tiles: every (stage, row tile, column block) exactly once, inside its
    # queue's range, GEMM-1 tiles before GEMM-2 tiles, and each group run column
    # block by column block with its row tiles back to back
    seen = set()
    for q in range(8):
        lo, n = int(qu[q, 0]), int(qu[q, 1])
        mine = tl[tl[:, 0] == q]
        assert len(mine) == n * (n1 + n2)
        assert np.all((mine[:, 2] >= lo) & (mine[:, 2] < lo + n))
        st = mine[:, 1]
        assert np.all(st[: n * n1] == 1) and np.all(st[n * n1:] == 2)
        for stage, nn, part in ((1, n1, mine[: n * n1]), (2, n2, mine[n * n1:])):
            assert np.all((part[:, 3] >= 0) & (part[:, 3] < nn))
            i = 0
            while i < len(part):
                f, s = gr[part[i, 2]]
                block = part[i:i + s * nn]
                want = [(int(f) + r, b) for b in range(nn) for r in range(s)]
                assert [(int(a), int(b)) for a, b in block[:, 2:4]] == want
                i += s * nn
            for t in part:
                key = (stage, int(t[2]), int(t[3]))
                assert key not in seen
                seen.add(key)
    assert len(seen) == x * (n1 + n2)


@pytest.mark.parametrize("M_t", [32, 128, 192])
@pytest.mark.parametrize("gmax", [1, 3, 8, 64])
def test_random_ragged_layouts(M_t, gmax):
    rng = np.random.default_rng(M_t * 100 + gmax)
    for _ in range(12):
        E = int(rng.integers(1, 65))
        counts = rng.integers(0, 900, size=E)
        counts[rng.random(E) < 0.25] = 0
        if rng.random() < 0.3:
            counts[int(rng.integers(0, E))] = int(rng.integers(2000, 5000))    # one hot expert
        n1, n2 = int(rng.integers(1, 7)), int(rng.integers(1, 7))
        _check(counts, _contiguous_offsets(counts), M_t, gmax, n1, n2)


def test_masked_offsets_and_edge_cases():
    # masked layout: fixed regions; single rows; empty op; one huge queue past the LDS cache
    _check(np.array([5, 0, 33, 1]), np.arange(4) * 64, 128, 8, 2, 3)
    _check(np.array([1]), np.array([0]), 192, 8, 1, 1)
    _check(np.zeros(7, np.int64), np.arange(7) * 32, 128, 8, 2, 2)
    big = np.full(40, 2000)
    _check(big, _contiguous_offsets(big), 32, 64, 2, 2)     # 2500 row tiles, queues of ~300 > cache
    hot_expert = np.array([3034] + [480] * 31)
    _check(hot_expert, _contiguous_offsets(hot_expert), 192, 8, 12, 12)


def test_claims_resolve_the_same_on_every_xcd():
    """moe_sched_layout returns -2 when a claim resolves differently through a
    workgroup's LDS cache than through memory; sizes around the cache width
    (64 row tiles per queue) must all agree."""
    for per_queue in (63, 64, 65, 127, 128):
        counts = np.full(8, per_queue * 32)
        _check(counts, _contiguous_offsets(counts), 32, 64, 1, 1)
