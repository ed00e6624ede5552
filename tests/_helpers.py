"""Shared test helpers: seeded inputs -> device specs, and the comparison rules.

Comparison rules (per the hot path's tolerances): routing and permutation
indices bit-exact; routing weights within 1e-6 relative; expert outputs and
the combined outputs per token (row) normwise relative error
||got - want||_2 / ||want||_2 <= 1e-2 for bf16 (3e-2 for fp8); rows whose
reference is exactly zero must be exactly zero."""
from __future__ import annotations

import numpy as np

import oracle
from workload import make_layer

BF16_TOL = 1e-2
FP8_TOL = 3e-2


def normwise_rel_err(got: np.ndarray, want: np.ndarray) -> float:
    got = np.asarray(got, dtype=np.float64)
    want = np.asarray(want, dtype=np.float64)
    nw = np.linalg.norm(want, axis=1)
    zero = nw == 0
    if np.any(zero):
        assert np.all(got[zero] == 0.0), "rows with an exactly-zero reference must be exactly zero"
    if np.all(zero):
        return 0.0
    return float(np.max(np.linalg.norm(got[~zero] - want[~zero], axis=1) / nw[~zero]))


def layer_specs(cfg, layer: int, device, phases=("prefill", "decode"), weights=None, lay=None, **ready):
    """(OpSpecs, LayerInputs) for one layer of a configuration, phases in order."""
    import torch

    from paper_2607_18002_amd.pipeline import LayerWeights, OpSpec, bf16_tensor
    from paper_2607_18002_amd import MOE_DECODE, MOE_PREFILL

    if lay is None:
        lay = make_layer(cfg, layer)
    if weights is None:
        weights = LayerWeights.from_numpy(lay.weights, cfg.H, cfg.I, device)
    specs = []
    for ph in lay.phases:
        if ph.phase not in phases:
            continue
        x = bf16_tensor(ph.x, device) if ph.x.dtype == np.uint16 else torch.from_numpy(ph.x).to(device)
        xs = torch.from_numpy(ph.x_scales).to(device) if ph.x_scales is not None else None
        specs.append(OpSpec(phase=MOE_PREFILL if ph.phase == "prefill" else MOE_DECODE, layer=layer,
                            logits=torch.from_numpy(ph.logits).to(device), x=x, x_scales=xs, weights=weights,
                            E_local=cfg.E_local, top_k=cfg.top_k, local_begin=cfg.local_begin,
                            **ready.get(ph.phase, {})))
    return specs, lay, weights


def oracle_for_phase(cfg, lay, ph, row_align: int, capacity: int):
    return oracle.moe_local_share(ph.logits, ph.x, lay.weights, cfg.top_k, cfg.local_begin, cfg.E_local,
                                  row_align, x_scales=ph.x_scales, capacity=capacity)
