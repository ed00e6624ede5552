"""Prefill/decode sharing of one MI355X: the adaptive persistent kernel against a
static CU partition and against time-sharing (the paper's single-GPU
microbenchmark, Evaluation "Effectiveness of APKs": concurrent prefill and
decode grouped GEMMs, decode arriving 10 us after prefill).

Mechanisms, all on the same two ops (one layer's prefill and decode share the
32 local experts' weights):
  * alone      : each op in its own persistent launch on the whole GPU
                 (the decode latency without load, the prefill time without load)
  * apk q=...  : both ops in ONE persistent launch, decode released 10 us after
                 the launch starts, decode quota q' workgroups (Eq. 4; fixed q or
                 adaptive with x*_moe)
  * partition  : both ops in one persistent launch with a static split (the
                 analogue of fixed SM partitions such as Green Contexts):
                 workgroups below q take only decode tiles, the others only
                 prefill tiles, and neither borrows the other's idle ones
                 (hipExtStreamCreateWithCUMask, the direct analogue, is refused
                 on the system this was measured on)
  * sequential : prefill then decode on one stream (time-sharing)
Reported per mechanism: decode op latency (its arrival, 10 us after the
prefill work started, to its last tile committed), prefill op latency (start
to done) and the makespan of both, from the kernels' device wall clock, and
each against the op alone.

Routing: Zipf-skewed logits over all 32 local experts (default), or, with
--active N, the paper's microbenchmark condition: both ops activate the same N
local experts (each token routes --local-slots of its k slots to them, round
robin, the rest to non-local experts).

    python -m paper_2607_18002_amd.sharing [--prefill 8192] [--decode 128] [--active 8]
"""
from __future__ import annotations

import argparse
from typing import Dict, List

import numpy as np

TICK_US = 0.01          # 100 MHz device wall clock


def _ops(T_p: int, T_d: int, H: int, I: int, E_g: int, E_l: int, k: int, seed: int, device, active: int = 0,
         local_slots: int = 1):
    """One layer's prefill and decode ops on shared random bf16 weights, with
    Zipf-skewed router logits (popularity rank r gets a bias of r^-1.1), or
    with `active` > 0, logits that route every token's `local_slots` local
    slots to the first `active` local experts."""
    import torch

    from ._lib import MOE_BF16, MOE_DECODE, MOE_PREFILL
    from .pipeline import LayerWeights, OpSpec

    g = torch.Generator(device=device).manual_seed(seed)
    gu = (torch.randn((E_l, 2 * I, H), generator=g, device=device) * 0.02).to(torch.bfloat16)
    wd = (torch.randn((E_l, H, I), generator=g, device=device) * 0.02).to(torch.bfloat16)
    w = LayerWeights(H, I, MOE_BF16, torch.empty_like(gu), torch.empty_like(wd))
    w.load(gu, wd)
    del gu, wd
    rank = torch.randperm(E_g, generator=torch.Generator().manual_seed(seed)).float() + 1.0
    bias = (rank ** -1.1).to(device)
    specs = {}
    for name, T, ph in (("prefill", T_p, MOE_PREFILL), ("decode", T_d, MOE_DECODE)):
        if active > 0:
            from .latency_model import routed_logits
            logits = torch.from_numpy(routed_logits(T, active, local_slots, E_g, E_l, k)).to(device)
        else:
            logits = torch.randn((T, E_g), generator=g, device=device) + bias[None, :]
        x = torch.randn((T, H), generator=g, device=device).to(torch.bfloat16)
        specs[name] = dict(phase=ph, layer=0, logits=logits, x=x, weights=w, E_local=E_l, top_k=k, local_begin=0)
    return specs, OpSpec


def _prepare(pipe) -> None:
    import torch
    pipe.route()
    pipe.permute()
    torch.cuda.synchronize()


def _since(st: np.ndarray, i: int, t_from: int) -> float:
    return (int(st["t_done"][i]) - t_from) * TICK_US


ARRIVE = int(10.0 / TICK_US)     # decode arrives 10 us after the prefill work starts


def run(T_p: int = 8192, T_d: int = 128, H: int = 3072, I: int = 1536, E_g: int = 256, E_l: int = 32, k: int = 8,
        quotas=(32, 64, 128), x_star: int = 0, partition_cus=(32, 64, 128), reps: int = 5,
        seed: int = 7, active: int = 0, local_slots: int = 1, q_max: int = 0, warmup: int = 20) -> List[Dict]:
    import torch

    from . import load_library
    from .pipeline import MoEPipeline

    load_library()
    dev = torch.device("cuda:0")
    n_cu = torch.cuda.get_device_properties(dev).multi_processor_count
    sp, OpSpec = _ops(T_p, T_d, H, I, E_g, E_l, k, seed, dev, active, local_slots)
    rows = []

    def med(vals):
        return float(np.median(vals))

    # warm-up (clocks and caches settle before the first measured mechanism)
    pw = MoEPipeline([OpSpec(**sp["prefill"]), OpSpec(**sp["decode"], release_after_ns=10_000)], fused_gather=True)
    _prepare(pw)
    for _ in range(warmup):
        pw.ffn()
    torch.cuda.synchronize()
    del pw

    # alone
    for name in ("prefill", "decode"):
        p = MoEPipeline([OpSpec(**sp[name])], fused_gather=True)
        _prepare(p)
        lat = []
        for _ in range(reps + 1):
            p.ffn()
            torch.cuda.synchronize()
            lat.append(_since(p.op_stats(), 0, p.kernel_t0()))
        rows.append(dict(mechanism=f"{name} alone (all {n_cu} CUs)", decode_us=med(lat[1:]) if name == "decode" else None,
                         prefill_us=med(lat[1:]) if name == "prefill" else None, makespan_us=med(lat[1:])))

    # APK: one launch, decode released 10 us after the start
    for q in quotas:
        specs = [OpSpec(**sp["prefill"]), OpSpec(**sp["decode"], release_after_ns=10_000)]
        p = MoEPipeline(specs, decode_quota_wg=q, decode_quota_max_wg=q_max, x_moe_expected=x_star, fused_gather=True)
        _prepare(p)
        d, pf, mk = [], [], []
        for _ in range(reps + 1):
            p.ffn()
            torch.cuda.synchronize()
            st, t0 = p.op_stats(), p.kernel_t0()
            d.append(_since(st, 1, t0 + ARRIVE))
            pf.append(_since(st, 0, t0))
            mk.append((max(int(st["t_done"][0]), int(st["t_done"][1])) - t0) * TICK_US)
        mode = "fixed" if x_star <= 0 else f"Eq. 4, x*_moe={x_star}"
        rows.append(dict(mechanism=f"APK, one launch, q={q} ({mode}), q'={int(st['quota'][1])}",
                         decode_us=med(d[1:]), prefill_us=med(pf[1:]), makespan_us=med(mk[1:])))

    # static partition: one launch, decode only on workgroups < P, prefill only on the rest
    for P in partition_cus:
        specs = [OpSpec(**sp["prefill"]), OpSpec(**sp["decode"], release_after_ns=10_000)]
        p = MoEPipeline(specs, decode_quota_wg=P, fused_gather=True, static_partition=True)
        _prepare(p)
        d, pf, mk = [], [], []
        for _ in range(reps + 1):
            p.ffn()
            torch.cuda.synchronize()
            st, t0 = p.op_stats(), p.kernel_t0()
            d.append(_since(st, 1, t0 + ARRIVE))
            pf.append(_since(st, 0, t0))
            mk.append((max(int(st["t_done"][0]), int(st["t_done"][1])) - t0) * TICK_US)
        rows.append(dict(mechanism=f"static partition: decode on {P} workgroups, prefill on {n_cu - P}",
                         decode_us=med(d[1:]), prefill_us=med(pf[1:]), makespan_us=med(mk[1:])))

    # sequential time-sharing: prefill, then decode, one stream
    pp = MoEPipeline([OpSpec(**sp["prefill"])], fused_gather=True)
    pd = MoEPipeline([OpSpec(**sp["decode"])], fused_gather=True)
    _prepare(pp)
    _prepare(pd)
    d, pf, mk = [], [], []
    for _ in range(reps + 1):
        pp.ffn()
        pd.ffn()
        torch.cuda.synchronize()
        spf, sd = pp.op_stats(), pd.op_stats()
        pf.append(_since(spf, 0, pp.kernel_t0()))
        # the decode op arrived 10 us after the prefill launch started and waited for it
        d.append(_since(sd, 0, pp.kernel_t0() + ARRIVE))
        mk.append((int(sd["t_done"][0]) - pp.kernel_t0()) * TICK_US)
    rows.append(dict(mechanism="sequential: prefill, then decode (one stream)", decode_us=med(d[1:]),
                     prefill_us=med(pf[1:]), makespan_us=med(mk[1:])))
    return rows


def main(argv=None) -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--prefill", type=int, default=8192)
    ap.add_argument("--decode", type=int, default=128)
    ap.add_argument("--x-star", type=int, default=0, help="x*_moe of Eq. (4); <= 0 for the fixed quota")
    ap.add_argument("--active", type=int, default=0, help="both ops activate this many local experts (0: Zipf)")
    ap.add_argument("--local-slots", type=int, default=1, help="with --active: local slots per token")
    ap.add_argument("--quotas", default="32,64,128")
    ap.add_argument("--qmax", type=int, default=0, help="Q_max of Eq. (4) in workgroups (0: half of them)")
    ap.add_argument("--partitions", default="32,64,128")
    args = ap.parse_args(argv)
    rows = run(T_p=args.prefill, T_d=args.decode, x_star=args.x_star, active=args.active,
               local_slots=args.local_slots, quotas=[int(v) for v in args.quotas.split(",")], q_max=args.qmax,
               partition_cus=[int(v) for v in args.partitions.split(",")])
    route = (f"{args.active} active local experts, {args.local_slots} local slot(s) per token" if args.active
             else "Zipf-skewed over 32 local experts")
    print(f"prefill {args.prefill} tokens + decode {args.decode} tokens, H 3072, I 1536, 32 of 256 experts, top-8, "
          f"bf16, {route}")
    alone_d = next(r["decode_us"] for r in rows if r["mechanism"].startswith("decode alone"))
    alone_p = next(r["prefill_us"] for r in rows if r["mechanism"].startswith("prefill alone"))
    print("| mechanism | decode op latency us | vs decode alone | prefill op latency us | vs prefill alone | makespan us |")
    print("|---|---|---|---|---|---|")
    f = lambda v: "-" if v is None else f"{v:.1f}"  # noqa: E731
    g = lambda v, base: "-" if v is None else f"{v / base:.2f}x"  # noqa: E731
    for r in rows:
        print(f"| {r['mechanism']} | {f(r['decode_us'])} | {g(r['decode_us'], alone_d)} | {f(r['prefill_us'])} | "
              f"{g(r['prefill_us'], alone_p)} | {f(r['makespan_us'])} |")
    return 0


if __name__ == "__main__":
    raise SystemExit(main())
