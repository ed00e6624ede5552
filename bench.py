#!/usr/bin/env python3
"""Benchmark of the routed-expert MoE hot path on one MI355X.

A step is one pass of the whole path over one batch: moe_topk_route and
moe_permute over every operation (one batched launch each; decode operations
use the masked layout by default, their rows placed by the routing launch), ONE
moe_grouped_ffn_persistent launch over all operations, and moe_combine over
every operation (one batched launch).  The default workload is
the mixed prefill+decode configuration: 4 layers x (8192 prefill + 1024 decode
tokens), 32 of 256 experts local, top-8, hidden 3072, expert intermediate
1536, bf16, in one persistent launch; decode layer 0 is released 10 us after
the launch starts, each later layer of a phase when that phase's previous
layer is done (+20 us for decode), decode quota 64 of 256 workgroups (the
configuration's 25% of the CUs).

Prints ONE JSON line.  value = routed-expert TFLOP/s of the whole step
(6*H*I flop per local routed row).  roofline = the persistent FFN kernel
against its bound (algorithmic bytes: the weights of every (layer, expert)
that receives a row, once per launch -- a layer's prefill and decode ops share
them -- plus the activation rows in and y_perm rows out; flops 6*H*I per row),
its mean duration over the timed steps from HIP events on its stream; traffic
= HBM bytes per launch from the committed rocprofv3 counter record when it was
taken on the current kernel sources, else null.  The timed launches carry the
per-tile trace (no round trip per tile); decode_tile_latency and the clock
the GEMM tiles ran at (shader clock counter over wall clock, reported with the
MFMA fraction at that clock) come from the last timed launch, and a launch
of the decode ops alone (same inputs and release chain) gives the latency
without prefill load.
cpu_baseline = the float64 CPU oracle over the whole workload, on this host's
cores; its outputs are then compared with the GPU's outputs of the last timed
step (parity: per-token normwise error and the whole-tensor figure).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

# The pipeline the benchmark times (tests build the same one from here).
DEFAULTS = dict(quota=64, decode_layout="masked", prefill_layout="contiguous", fused_combine=False,
                group_row_tiles=0, gather="fused", prefill_tile_rows=0)

HBM_PEAK_GBS = 8000.0
MFMA_PEAK_TFLOPS = {"bf16": 2500.0, "fp8": 5000.0}
NOMINAL_CLOCK_GHZ = 2.4          # peak engine clock the dense MFMA peaks are quoted at
TICK_NS = 10.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", type=int, default=4, help="workload configuration (1-5); default 4")
    ap.add_argument("--quota", type=int, default=DEFAULTS["quota"], help="decode quota q in workgroups")
    ap.add_argument("--decode-layout", choices=["masked", "contiguous"], default=DEFAULTS["decode_layout"],
                    help="masked: decode ops' rows placed by routing in per-expert regions (no permute pass); "
                         "contiguous: permuted like prefill")
    ap.add_argument("--prefill-layout", choices=["masked", "contiguous"], default=DEFAULTS["prefill_layout"],
                    help="the same choice for prefill ops")
    ap.add_argument("--fused-combine", action="store_true",
                    help="combine tiles inside the persistent kernel instead of a separate combine launch")
    ap.add_argument("--group-row-tiles", type=int, default=0,
                    help="most row tiles of one expert that share each weight slice fetch (0 = library default)")
    ap.add_argument("--gather", choices=("fused", "copy"), default="fused",
                    help="GEMM-1 reads x rows through row_to_assign (fused) or from the permuted copy x_perm")
    ap.add_argument("--prefill-tile-rows", type=int, choices=(0, 128, 192), default=DEFAULTS["prefill_tile_rows"],
                    help="128: bf16 prefill ops run 128-row tiles (shorter preemption waits); 0/192: 192-row tiles")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--dump-trace", default=None, help="write the traced launch's per-tile records (.npy)")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="after the run, copy this many MiB device to device 3 times and stream-read as many "
                         "3 times (counter calibration: kernels of known bytes)")
    ap.add_argument("--no-peaks", action="store_true", help="skip the measured-peak microbenchmarks")
    return ap.parse_args()


def build_specs(cfg, dev):
    from paper_2607_18002_amd import MOE_DECODE, MOE_PREFILL
    from paper_2607_18002_amd.pipeline import LayerWeights, OpSpec, bf16_tensor
    from workload import make_layer
    import torch

    specs, layers = [], []
    prev = {"prefill": -1, "decode": -1}
    for layer in range(cfg.n_layers):
        lay = make_layer(cfg, layer)
        w = LayerWeights.from_numpy(lay.weights, cfg.H, cfg.I, dev)
        for ph in lay.phases:
            x = bf16_tensor(ph.x, dev) if ph.x.dtype == np.uint16 else torch.from_numpy(ph.x).to(dev)
            xs = torch.from_numpy(ph.x_scales).to(dev) if ph.x_scales is not None else None
            decode = ph.phase == "decode"
            ready = dict(release_after_ns=-1, depends_on_op=prev[ph.phase], gap_ns=0)
            if decode and layer == 0 and cfg.prefill_tokens > 0:
                ready["release_after_ns"] = 10_000
            if decode and layer > 0:
                ready["gap_ns"] = 20_000
            prev[ph.phase] = len(specs)
            specs.append(OpSpec(phase=MOE_DECODE if decode else MOE_PREFILL, layer=layer,
                                logits=torch.from_numpy(ph.logits).to(dev), x=x, x_scales=xs, weights=w,
                                E_local=cfg.E_local, top_k=cfg.top_k, local_begin=cfg.local_begin, **ready))
        layers.append(lay)
        del lay
    return specs, layers


def pipeline_kwargs(quota=DEFAULTS["quota"], decode_layout=DEFAULTS["decode_layout"],
                    prefill_layout=DEFAULTS["prefill_layout"], fused_combine=DEFAULTS["fused_combine"],
                    group_row_tiles=DEFAULTS["group_row_tiles"], gather=DEFAULTS["gather"],
                    prefill_tile_rows=DEFAULTS["prefill_tile_rows"]):
    """MoEPipeline arguments of a benchmark configuration (the masked layouts
    need the fused gather)."""
    fused = gather == "fused"
    return dict(decode_quota_wg=quota, fused_gather=fused, fused_combine=fused_combine,
                masked_decode=decode_layout == "masked" and fused, masked_prefill=prefill_layout == "masked" and fused,
                group_row_tiles=group_row_tiles, prefill_tile_rows=prefill_tile_rows)


def tile_clock(tr):
    """Shader clock the GEMM tiles of a traced launch ran at (GHz, p10/p50/p90):
    shader clock counter over wall-clock ticks (100 MHz) per tile."""
    tr = tr[(tr["stage"] < 3) & (tr["t_end"] > tr["t_start"])]
    if len(tr) == 0:
        return None
    f = (tr["c_end"] - tr["c_start"]).astype(np.float64) / ((tr["t_end"] - tr["t_start"]).astype(np.float64) * 10.0)
    return [round(float(np.percentile(f, q)), 3) for q in (10, 50, 90)]


def algorithmic_work(pipe, cfg):
    """flops and HBM bytes the method itself must move, per persistent launch.

    Weights: every (layer, local expert) that receives at least one row, once
    per launch (the prefill and decode ops of a layer share the layer's
    experts).  Activations: each routed row read once, its y_perm row written
    once.  Also returns the weight bytes counted once per op instead (what a
    schedule that never shares a fetch between the phases must move)."""
    b_w = 1 if cfg.dtype == "fp8" else 2
    b_x = 1 if cfg.dtype == "fp8" else 2
    w_expert = 3.0 * cfg.H * cfg.I * b_w
    if cfg.dtype == "fp8":
        w_expert += 3.0 * (cfg.H // 128) * (cfg.I // 128) * 4
    flops = 0.0
    act_bytes = 0.0
    per_op_w = 0.0
    rows_total = 0
    active_by_layer = {}
    for b in pipe.bufs:
        counts = b.counts.cpu().numpy()
        R = int(counts.sum())
        rows_total += R
        flops += 6.0 * cfg.H * cfg.I * R
        act_bytes += R * cfg.H * (b_x + 2) + (R * (cfg.H // 128) * 4 if cfg.dtype == "fp8" else 0)
        per_op_w += int(np.count_nonzero(counts)) * w_expert
        lay = active_by_layer.setdefault(b.spec.layer, np.zeros(len(counts), dtype=bool))
        lay |= counts > 0
    unique_w = sum(int(v.sum()) for v in active_by_layer.values()) * w_expert
    return flops, unique_w + act_bytes, rows_total, per_op_w + act_bytes


def decode_latency(pipe, specs):
    """Decode latency figures from one traced launch, in microseconds.

    release(op) = the time the op became eligible (launch start + its delay,
    or its predecessor's completion + gap).  Tile latency = t_end - release;
    preemption wait = first tile start - release; op latency = last tile end -
    release."""
    st = pipe.op_stats()
    tr = pipe.trace_records()
    t0 = pipe.kernel_t0()
    lat, waits, op_lat, parts = [], [], [], []
    for i, s in enumerate(specs):
        if s.phase != 1:
            continue
        if s.release_after_ns >= 0:
            rel = t0 + s.release_after_ns / TICK_NS
        elif s.depends_on_op >= 0:
            rel = float(st["t_done"][s.depends_on_op]) + s.gap_ns / TICK_NS
        else:
            rel = float(t0)
        mine = tr[tr["op"] == i]
        if len(mine) == 0:
            continue
        us = lambda t: (t.astype(np.float64) - rel) * TICK_NS / 1000.0  # noqa: E731
        lat.extend(us(mine["t_end"]).tolist())
        waits.append(float(us(mine["t_start"]).min()))
        # the wait in parts: release seen at a boundary, instantiation, first tile start
        parts.append([round(float((st["t_seen"][i] - rel) * TICK_NS / 1000.0), 1),
                      round(float((st["t_ready"][i] - st["t_seen"][i]) * TICK_NS / 1000.0), 1),
                      round(float(us(mine["t_start"]).min() - (st["t_ready"][i] - rel) * TICK_NS / 1000.0), 1)])
        op_lat.append(float(us(mine["t_end"]).max()))
    tiles = {}
    for ph, pname in ((0, "prefill"), (1, "decode")):
        ops_ph = [i for i, s in enumerate(specs) if s.phase == ph]
        for stage in (1, 2):
            sel = np.isin(tr["op"], ops_ph) & (tr["stage"] == stage)
            if not np.any(sel):
                continue
            d = (tr["t_end"][sel].astype(np.float64) - tr["t_start"][sel]) * TICK_NS / 1000.0
            tiles[f"{pname}_gemm{stage}"] = {"n": int(sel.sum()),
                                             **{f"p{q}_us": round(float(np.percentile(d, q)), 2) for q in (10, 50, 90, 99)},
                                             "max_us": round(float(d.max()), 2)}
    if not lat:
        return {"tile_duration": tiles}
    pre = np.isin(tr["op"], [i for i, s in enumerate(specs) if s.phase == 0])
    ptd = (tr["t_end"][pre].astype(np.float64) - tr["t_start"][pre]) * TICK_NS / 1000.0
    return {"tile_duration": tiles,
            "tile_p50_us": round(float(np.percentile(lat, 50)), 2),
            "tile_p99_us": round(float(np.percentile(lat, 99)), 2),
            "preempt_wait_max_us": round(max(waits), 2), "preempt_wait_mean_us": round(float(np.mean(waits)), 2),
            "preempt_wait_parts_us": {"per_decode_op": parts,
                                      "legend": "release->seen at a tile boundary, instantiation, ->first tile start"},
            "decode_op_latency_us": [round(v, 1) for v in op_lat],
            "prefill_tile_max_us": round(float(ptd.max()), 2) if len(ptd) else None,
            "prefill_tile_p50_us": round(float(np.percentile(ptd, 50)), 2) if len(ptd) else None}


def cpu_baseline(cfg, layers, outputs=None):
    """The oracle as it stands, on the same workload: every operation of every
    layer (all tokens, every step of the path), on this host's cores.  When
    `outputs` (the oracle's y per op, in op order) is a list, it is filled."""
    import oracle
    try:
        from threadpoolctl import threadpool_info
        cores = max([p.get("num_threads", 1) for p in threadpool_info()] + [1])
    except Exception:  # pragma: no cover
        cores = len(os.sched_getaffinity(0))
    flops, rows, dt = 0.0, 0, 0.0
    for lay in layers:
        for ph in lay.phases:
            t = time.perf_counter()
            res = oracle.moe_local_share(ph.logits, ph.x, lay.weights, cfg.top_k, cfg.local_begin, cfg.E_local,
                                         128, x_scales=ph.x_scales)
            dt += time.perf_counter() - t
            if outputs is not None:
                outputs.append(res["y"])
            R = int(res["perm"].counts.sum())
            rows += R
            flops += 6.0 * cfg.H * cfg.I * R
    desc = " + ".join(f"{ph.T} {ph.phase}" for ph in layers[0].phases)
    return {"value": round(flops / dt / 1e12, 5), "unit": "TFLOP/s", "cores": int(cores), "kind": "oracle",
            "sample": f"the whole workload: {cfg.n_layers} layer(s) x ({desc} tokens), {rows} local rows, every "
                      f"step of the path, float64 numpy, {dt:.1f} s"}


def output_parity(pipe, want, tol):
    """GPU y of every op against the oracle's: the largest per-token normwise
    relative error (tokens whose oracle output is exactly zero must be exactly
    zero on the GPU) and the whole-tensor max|y - y_ref| / max|y_ref|."""
    worst, whole, zeros_ok = 0.0, 0.0, True
    for b, ref in zip(pipe.bufs, want):
        y = b.y.float().cpu().numpy().astype(np.float64)
        nw = np.linalg.norm(ref, axis=1)
        z = nw == 0
        zeros_ok &= bool(np.all(y[z] == 0.0))
        if np.any(~z):
            worst = max(worst, float(np.max(np.linalg.norm(y[~z] - ref[~z], axis=1) / nw[~z])))
        m = float(np.abs(ref).max())
        if m > 0:
            whole = max(whole, float(np.abs(y - ref).max()) / m)
    return {"per_token_normwise_max": float(f"{worst:.3e}"), "whole_tensor_max_rel": float(f"{whole:.3e}"),
            "zero_tokens_exact": zeros_ok, "tolerance": tol, "ok": bool(worst <= tol and zeros_ok)}


def traffic_record(workload):
    """HBM bytes per launch recorded by rocprofv3 counters for this workload,
    or None when no record exists or the kernel sources changed since."""
    from paper_2607_18002_amd.build import ffn_kernel_hash
    path = os.path.join(ROOT, "profiles", f"apk_kernel_traffic_{workload}.md")
    if not os.path.exists(path):
        return None
    kv = {}
    with open(path) as f:
        for line in f:
            if " = " in line:
                k, v = line.split(" = ", 1)
                kv[k.strip()] = v.strip()
    if kv.get("source_hash") != ffn_kernel_hash() or kv.get("workload") != workload:
        return None
    return float(kv["traffic_bytes_per_launch"])


def phase_subset(specs, phase):
    """The ops of one phase alone, with dependencies renumbered (same inputs)."""
    import dataclasses
    keep = [i for i, s in enumerate(specs) if s.phase == phase]
    remap = {old: new for new, old in enumerate(keep)}
    out = []
    for i in keep:
        s = specs[i]
        dep = remap.get(s.depends_on_op, -1)
        out.append(dataclasses.replace(s, depends_on_op=dep))
    return out


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one MI355X: this path has no multi-GPU mode (run with --gpus 1)", file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_2607_18002_amd import load_library
    from paper_2607_18002_amd.pipeline import MoEPipeline
    from workload import CONFIGS

    load_library()
    dev = torch.device("cuda:0")
    cfg = CONFIGS[args.config]
    t_gen = time.perf_counter()
    specs, layers = build_specs(cfg, dev)
    t_gen = time.perf_counter() - t_gen
    pkw = pipeline_kwargs(args.quota, args.decode_layout, args.prefill_layout, args.fused_combine,
                          args.group_row_tiles, args.gather, args.prefill_tile_rows)
    # the per-tile trace costs no round trip (each workgroup writes its own
    # block), so the timed launches carry it: the last one gives the decode
    # latency and clock figures in the timed loop's own steady state
    pipe = MoEPipeline(specs, trace_capacity=1 << 18, **pkw)
    stream = torch.cuda.current_stream()

    for _ in range(args.warmup):
        pipe.run()
    torch.cuda.synchronize()
    err, status = pipe.statuses()
    if err or status:
        raise SystemExit(f"device status after warmup: permute={err} ffn={status}")

    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for i in range(args.steps):
        pipe.route()
        pipe.permute()
        ev[i][0].record(stream)
        pipe.ffn()
        ev[i][1].record(stream)
        pipe.combine()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start
    ffn_all = np.array([a.elapsed_time(b) for a, b in ev])
    ffn_ms = float(np.mean(ffn_all))
    ms_step = wall * 1000.0 / args.steps

    flops, abytes, rows, abytes_per_op = algorithmic_work(pipe, cfg)
    traced = pipe                                      # its last timed launch
    if args.dump_trace:
        np.save(args.dump_trace, traced.trace_records())
        np.save(args.dump_trace.replace(".npy", "_stats.npy"), traced.op_stats())
    err, status = traced.statuses()
    if err or status:
        raise SystemExit(f"device status of the traced launch: permute={err} ffn={status}")
    lat = decode_latency(traced, specs)
    clock = tile_clock(traced.trace_records())
    # the decode ops alone (same inputs, same release chain): the latency without prefill load
    excl = None
    dec_specs = phase_subset(specs, 1)
    if lat is not None and "tile_p99_us" in lat and dec_specs and len(dec_specs) < len(specs):
        alone = MoEPipeline(dec_specs, trace_capacity=1 << 16, **pkw)
        alone.run()
        alone.run()
        torch.cuda.synchronize()
        err, status = alone.statuses()
        if err or status:
            raise SystemExit(f"device status of the decode-only launch: permute={err} ffn={status}")
        excl = decode_latency(alone, dec_specs)
        del alone
        lat["exclusive_tile_p50_us"] = excl["tile_p50_us"]
        lat["exclusive_tile_p99_us"] = excl["tile_p99_us"]
        lat["exclusive_decode_op_latency_us"] = excl["decode_op_latency_us"]
        lat["p99_ratio_loaded_vs_exclusive"] = round(lat["tile_p99_us"] / excl["tile_p99_us"], 3)
    if args.calib_copy_mib > 0:
        n = args.calib_copy_mib << 20
        src = torch.empty(n, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
        from paper_2607_18002_amd import peaks
        peaks.stream_read_gbs(gib=args.calib_copy_mib / 1024.0, reps=1)   # 3 launches of known read bytes
        torch.cuda.synchronize()

    dtype = cfg.dtype
    t_mfma = flops / (MFMA_PEAK_TFLOPS[dtype] * 1e12)
    t_hbm = abytes / (HBM_PEAK_GBS * 1e9)
    bound = "hbm" if t_hbm >= t_mfma else "mfma"
    if bound == "hbm":
        ach = abytes / (ffn_ms * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": round(ach, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(ach / HBM_PEAK_GBS, 4), "traffic": None}
    else:
        ach = flops / (ffn_ms * 1e-3) / 1e12
        roof = {"bound": "mfma", "achieved": round(ach, 1), "peak": MFMA_PEAK_TFLOPS[dtype], "unit": "TFLOP/s",
                "frac": round(ach / MFMA_PEAK_TFLOPS[dtype], 4), "traffic": None}
    tb = traffic_record(cfg.name)
    roof["traffic"] = tb
    if tb is not None:
        roof["traffic_vs_alg_bytes"] = round(tb / abytes, 3)
    roof["kernel"] = "apk_kernel (moe_grouped_ffn_persistent)"
    roof["kernel_ms"] = round(ffn_ms, 4)
    roof["kernel_ms_p10_p50_p90"] = [round(float(np.percentile(ffn_all, q)), 4) for q in (10, 50, 90)]
    roof["alg_bytes"] = abytes
    roof["alg_bytes_weights_once_per_op"] = abytes_per_op
    roof["alg_flops"] = flops
    roof["achieved_tflops"] = round(flops / (ffn_ms * 1e-3) / 1e12, 2)
    roof["frac_mfma"] = round(flops / (ffn_ms * 1e-3) / 1e12 / MFMA_PEAK_TFLOPS[dtype], 4)
    roof["frac_hbm"] = round(abytes / (ffn_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)
    if clock is not None:
        # the MFMA peak scales with the shader clock (2.5 PFLOP/s bf16 dense is quoted at 2.4 GHz)
        roof["tile_clock_ghz_p10_p50_p90"] = clock
        roof["frac_mfma_at_tile_clock"] = round(roof["frac_mfma"] * NOMINAL_CLOCK_GHZ / clock[1], 4)

    if not args.no_peaks:
        from paper_2607_18002_amd import peaks
        meas = peaks.measure()
        roof["measured_peaks"] = meas
        roof["frac_of_measured_mfma"] = round(roof["achieved_tflops"] / meas[f"mfma_{dtype}_tflops"], 4)
        roof["frac_of_measured_hbm"] = round(abytes / (ffn_ms * 1e-3) / 1e9 / meas["hbm_read_gbs"], 4)
        if dtype == "bf16":
            roof["vs_vendor_dense_gemm"] = round(roof["achieved_tflops"] / meas["vendor_gemm_bf16_16384x3072x3072_tflops"], 4)

    cpu = None
    parity = None
    if not args.no_cpu_baseline:
        want = []
        cpu = cpu_baseline(cfg, layers, want)
        parity = output_parity(pipe, want, 3e-2 if dtype == "fp8" else 1e-2)
        del want

    out = {
        "metric": "routed-expert TFLOP/s + HBM GB/s per MI355X (mixed P/D); decode p99 tile latency",
        "value": round(flops / (ms_step * 1e-3) / 1e12, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f8e4m3" if dtype == "fp8" else "bf16",
        "data": "synthetic (seeded; random-init expert weights, Zipf-skewed router logits)",
        "config": {"workload": cfg.name, "config_id": cfg.cfg_id, "layers": cfg.n_layers,
                   "prefill_tokens": cfg.prefill_tokens, "decode_tokens": cfg.decode_tokens,
                   "experts_local": cfg.E_local, "experts_global": cfg.E_global, "top_k": cfg.top_k,
                   "hidden": cfg.H, "intermediate": cfg.I, "decode_quota_wg": args.quota,
                   "group_row_tiles": args.group_row_tiles, "prefill_tile_rows": args.prefill_tile_rows or 192,
                   "gather": args.gather, "combine": "fused" if args.fused_combine else "separate",
                   "decode_layout": "masked" if pkw["masked_decode"] else "contiguous",
                   "prefill_layout": "masked" if pkw["masked_prefill"] else "contiguous", "local_rows": rows},
        "hbm_gbps_alg": round(abytes / (ffn_ms * 1e-3) / 1e9, 1),
        "ffn_tflops": round(flops / (ffn_ms * 1e-3) / 1e12, 2),
        "decode_tile_latency": lat,
        "roofline": roof,
        "cpu_baseline": cpu,
        "parity_vs_oracle": parity,
        "input_gen_s": round(t_gen, 1),
    }
    print(json.dumps(out))


if __name__ == "__main__":
    main()
