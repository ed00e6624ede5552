"""What the persistent tile scheduler costs against the same tiles launched as
plain grids (the paper's Evaluation, "Overhead of Tile-Level Scheduling":
its adaptive persistent kernel against plain grouped-GEMM launches, the
contiguous layout swept over the per-expert batch, the masked layout over
the number of active experts).

One op per measurement, routed so that `active` local experts receive
near-equal rows; the persistent launch (moe_grouped_ffn_persistent) and the
plain grids (moe_grouped_ffn_plain: planning, GEMM-1 and GEMM-2 launches) are
timed with HIP events on one stream, median of `reps`.

    python -m paper_2607_18002_amd.overhead
"""
from __future__ import annotations

import argparse

import numpy as np


def _time(fn, reps):
    import torch
    s = torch.cuda.current_stream()
    fn()
    torch.cuda.synchronize()
    out = []
    for _ in range(reps):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(s)
        fn()
        b.record(s)
        torch.cuda.synchronize()
        out.append(a.elapsed_time(b) * 1000.0)
    return float(np.median(out))


def run(points, phase, H=3072, I=1536, E_g=256, E_l=32, k=8, reps=10, seed=0):
    import torch

    from . import load_library
    from ._lib import MOE_BF16, MOE_DECODE, MOE_PREFILL
    from .latency_model import routed_logits
    from .pipeline import LayerWeights, MoEPipeline, OpSpec

    load_library()
    dev = torch.device("cuda:0")
    g = torch.Generator(device=dev).manual_seed(seed)
    gu = (torch.randn((E_l, 2 * I, H), generator=g, device=dev) * 0.02).to(torch.bfloat16)
    wd = (torch.randn((E_l, H, I), generator=g, device=dev) * 0.02).to(torch.bfloat16)
    w = LayerWeights(H, I, MOE_BF16, torch.empty_like(gu), torch.empty_like(wd))
    w.load(gu, wd)
    del gu, wd
    ph = MOE_DECODE if phase == "decode" else MOE_PREFILL
    rows = []
    for T, active in points:
        logits = torch.from_numpy(routed_logits(T, active, 1, E_g, E_l, k)).to(dev)
        x = torch.randn((T, H), generator=g, device=dev).to(torch.bfloat16)
        spec = OpSpec(phase=ph, layer=0, logits=logits, x=x, weights=w, E_local=E_l, top_k=k)
        pipe = MoEPipeline([spec], fused_gather=True, masked_decode=phase == "decode")
        pipe.route()
        pipe.permute()
        torch.cuda.synchronize()
        t_apk = _time(pipe.ffn, reps)
        t_plain = _time(pipe.ffn_plain, reps)
        assert pipe.statuses() == (0, 0)
        # the persistent launch in parts, from its device wall clock (10 ns ticks)
        pipe.ffn()
        torch.cuda.synchronize()
        st, t0 = pipe.op_stats(), pipe.kernel_t0()
        us = lambda a, b: (int(a) - int(b)) / 100.0  # noqa: E731
        parts = (us(st["t_seen"][0], t0), us(st["t_ready"][0], st["t_seen"][0]), us(st["t_first"][0], st["t_ready"][0]),
                 us(st["t_done"][0], st["t_first"][0]))
        rows.append(dict(tokens=T, active=active, rows_per_expert=T // active, apk_us=t_apk, plain_us=t_plain,
                         overhead=t_apk / t_plain - 1.0, parts=parts))
        del pipe
    return rows


def main(argv=None) -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--reps", type=int, default=10)
    args = ap.parse_args(argv)
    sweeps = {
        "prefill (contiguous layout), 32 active experts, rows per expert swept":
            ("prefill", [(32 * m, 32) for m in (64, 128, 256, 512, 1024, 2048)]),
        "decode (masked layout), 128 tokens, active experts swept":
            ("decode", [(128, a) for a in (1, 2, 4, 8, 16, 32)]),
    }
    for title, (phase, pts) in sweeps.items():
        rows = run(pts, phase, reps=args.reps)
        print(f"{title}; H 3072, I 1536, bf16, one local slot per token")
        print("| tokens | active experts | rows per expert | persistent us | plain grids us | overhead | "
              "persistent: start->seen / instantiation / ->first tile / tiles us |")
        print("|---|---|---|---|---|---|---|")
        for r in rows:
            print(f"| {r['tokens']} | {r['active']} | {r['rows_per_expert']} | {r['apk_us']:.1f} | {r['plain_us']:.1f} | "
                  f"{100 * r['overhead']:+.1f}% | " + " / ".join(f"{v:.1f}" for v in r["parts"]) + " |")
    return 0


if __name__ == "__main__":
    raise SystemExit(main())
