"""Host arithmetic of the tile-aware latency model: Eq. (3) footprint against
the oracle's, the least-squares fits recovering known coefficients, and the
sweep's routing construction (checked with the oracle's router)."""
import numpy as np

import oracle
from paper_2607_18002_amd import latency_model as lm


def test_footprint_matches_eq3():
    rng = np.random.default_rng(5)
    for _ in range(200):
        counts = rng.integers(0, 900, int(rng.integers(1, 40))) * (rng.random() < 0.9)
        for mt in (32, 64, 128, 192):
            assert lm.footprint(counts, mt) == oracle.x_moe(counts, mt)
    assert lm.footprint([0, 0, 0], 128) == 0
    assert lm.footprint([1, 128, 129], 128) == 1 + 1 + 2


def test_fit_line_recovers_a_line():
    x = np.arange(1, 40, dtype=np.float64)
    a, b, r2 = lm.fit_line(x, 0.012 + 0.0034 * x)
    assert abs(a - 0.012) < 1e-12 and abs(b - 0.0034) < 1e-12 and abs(r2 - 1.0) < 1e-12
    noisy = 0.012 + 0.0034 * x + np.where(np.arange(x.size) % 2, 1e-4, -1e-4)
    a, b, r2 = lm.fit_line(x, noisy)
    assert abs(b - 0.0034) < 1e-5 and r2 > 0.999


def test_fit_full_recovers_the_general_form():
    rng = np.random.default_rng(1)
    x = rng.integers(1, 64, 50).astype(np.float64)
    s = rng.integers(1, 4096, 50).astype(np.float64)
    t = 3.0 + 0.5 * x + 1e-3 * x * s + 2e-7 * x * s * s
    coef = lm.fit_full(x, s, t)
    assert np.allclose(coef, (3.0, 0.5, 1e-3, 2e-7), rtol=1e-6, atol=1e-9)


def test_sweep_routing_hits_the_requested_experts():
    for T, act, ls in ((64, 4, 1), (100, 8, 2), (33, 32, 1), (5, 1, 1)):
        L = lm.routed_logits(T, act, ls, 256, 32, 8)
        ids, w = oracle.route(L, 8, 0, 32)
        local = ids[ids >= 0]
        assert local.size == T * ls
        assert set(np.unique(local).tolist()) == set(range(min(act, T * ls)))
        counts = np.bincount(local, minlength=32)
        nz = counts[counts > 0]
        assert nz.max() - nz.min() <= 1                     # near-equal rows per active expert
