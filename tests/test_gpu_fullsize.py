"""Full-size parity of the benchmarked path against the CPU oracle, every
token and every routed row.

The pipeline is built exactly as bench.py builds it (same inputs, release
chain, quota, layouts, gather and combine), run twice on the same buffers,
then compared with the float64 oracle:

* routing ids bit-exact, weights within 1e-6 relative;
* permutation indices bit-exact against the oracle's layout of the same kind
  (contiguous segments, or the masked layout's fixed regions);
* every routed row's expert output (y_perm) and every token's output y within
  the per-row / per-token normwise bound (1e-2 bf16, 3e-2 fp8 against the
  unquantized oracle); tokens whose oracle output is exactly zero are exactly
  zero; the whole-tensor max|y - y_ref| / max|y_ref| is printed and bounded
  the same way."""
import os
import sys

import numpy as np
import pytest

import oracle
from _helpers import BF16_TOL, FP8_TOL, normwise_rel_err
from workload import CONFIGS

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)
import bench  # noqa: E402


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2607_18002_amd import load_library
    load_library()
    return torch.device("cuda:0")


_CACHE = {}


def _inputs(cfg_id, dev):
    """Device specs, host layer inputs and the oracle's results of every op
    (contiguous layout: the expert outputs do not depend on the layout), kept
    for the configuration's other cases."""
    if cfg_id in _CACHE:
        return _CACHE[cfg_id]
    _CACHE.clear()
    cfg = CONFIGS[cfg_id]
    specs, layers = bench.build_specs(cfg, dev)
    refs = []
    for lay in layers:
        for ph in lay.phases:
            r = oracle.moe_local_share(ph.logits, ph.x, lay.weights, cfg.top_k, cfg.local_begin, cfg.E_local, 32,
                                       x_scales=ph.x_scales)
            refs.append(dict(ids=r["ids"], w=r["w"], a2r=r["perm"].assign_to_row, y_perm=r["y_perm"], y=r["y"]))
    _CACHE[cfg_id] = (cfg, specs, layers, refs)
    return _CACHE[cfg_id]


CASES = [
    (4, {}),                                   # the benchmark's default configuration
    (4, {"fused_combine": True}),
    (4, {"prefill_layout": "masked"}),
    (4, {"decode_layout": "contiguous", "gather": "copy"}),
    (2, {}),
    (3, {}),
    (3, {"prefill_layout": "masked"}),
    (5, {}),
]


@pytest.mark.parametrize("cfg_id,kw", CASES, ids=[f"cfg{c}-" + ("-".join(f"{k}={v}" for k, v in kw.items()) or "bench")
                                                  for c, kw in CASES])
def test_full_size_every_token(dev, cfg_id, kw):
    from paper_2607_18002_amd.pipeline import MoEPipeline
    cfg, specs, layers, refs = _inputs(cfg_id, dev)
    print(f"\nfull-size cfg{cfg_id} {kw}", flush=True)
    pipe = MoEPipeline(specs, **bench.pipeline_kwargs(**kw))
    for b in pipe.bufs:
        b.y.fill_(7.0)                                   # every output element must be written
    for _ in range(2):
        pipe.run()
    torch.cuda.synchronize()
    assert pipe.statuses() == (0, 0)
    tol = FP8_TOL if cfg.dtype == "fp8" else BF16_TOL
    k = cfg.top_k
    worst_row, worst_tok, worst_whole = 0.0, 0.0, 0.0
    for i, b in enumerate(pipe.bufs):
        ref = refs[i]
        np.testing.assert_array_equal(b.topk_ids.cpu().numpy(), ref["ids"])
        np.testing.assert_allclose(b.topk_w.cpu().numpy(), ref["w"], rtol=1e-6, atol=1e-9)
        a2r = b.assign_to_row.cpu().numpy()
        r2a = b.row_to_assign.cpu().numpy()
        counts = b.counts.cpu().numpy()
        offsets = b.offsets.cpu().numpy()
        if b.slots > 0:
            p = oracle.permute_masked(ref["ids"], cfg.E_local, b.slots)
            for e in range(cfg.E_local):
                lo = int(p.offsets[e])
                np.testing.assert_array_equal(r2a[lo:lo + p.counts[e]], p.row_to_assign[lo:lo + p.counts[e]])
        else:
            p = oracle.permute(ref["ids"], cfg.E_local, b.row_align, capacity=b.capacity)
            used = int(p.offsets[-1])
            np.testing.assert_array_equal(r2a[:used], p.row_to_assign[:used])
        np.testing.assert_array_equal(counts, p.counts)
        np.testing.assert_array_equal(offsets, p.offsets)
        np.testing.assert_array_equal(a2r, p.assign_to_row)
        # every routed row: the GPU row of assignment a against the oracle's row of a
        loc = np.nonzero(a2r >= 0)[0]
        got_rows = b.y_perm[torch.from_numpy(a2r[loc]).long().to(dev)].float().cpu().numpy()
        err_row = normwise_rel_err(got_rows, ref["y_perm"][ref["a2r"][loc]])
        y = b.y.float().cpu().numpy()
        err_tok = normwise_rel_err(y, ref["y"])
        m = float(np.abs(ref["y"]).max())
        whole = float(np.abs(y - ref["y"]).max()) / m if m > 0 else float(np.abs(y).max())
        print(f"  op {i} (layer {b.spec.layer}, {'decode' if b.spec.phase else 'prefill'}): T={b.T} rows={len(loc)} "
              f"y_perm row max {err_row:.3e}  y token max {err_tok:.3e}  whole-tensor {whole:.3e}", flush=True)
        worst_row, worst_tok, worst_whole = max(worst_row, err_row), max(worst_tok, err_tok), max(worst_whole, whole)
        assert err_row <= tol, (i, err_row)
        assert err_tok <= tol, (i, err_tok)
        assert whole <= tol, (i, whole)
    print(f"  worst: y_perm row {worst_row:.3e}, y token {worst_tok:.3e}, whole-tensor {worst_whole:.3e} "
          f"(bound {tol})", flush=True)
