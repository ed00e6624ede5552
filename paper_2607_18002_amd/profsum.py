"""Summaries of rocprofv3 databases for the persistent FFN kernel.

    python -m paper_2607_18002_amd.profsum stats DB --skip W --take K --cmd "..."
    python -m paper_2607_18002_amd.profsum traffic --fetch DB1 --write DB2 --skip W --take K \
        --copy-bytes B --workload NAME --cmd-fetch "..." --cmd-write "..."
    python -m paper_2607_18002_amd.profsum counters DB --counters A,B --skip W --take K --cmd "..."

``stats`` reads a ``rocprofv3 --kernel-trace --stats`` database and prints
per-kernel call counts and durations, plus the average of the persistent
kernel's dispatches number W .. W+K-1 (the timed region of bench.py, which
launches W warm-up steps first).

``traffic`` reads two ``rocprofv3 --pmc`` databases, one with FETCH_SIZE and
one with WRITE_SIZE (KiB per dispatch).  Each counter is calibrated on a plain
device-to-device copy of B bytes in the same run (it reads B and writes B), and
the persistent kernel's timed-region average is scaled by that factor.  The
output carries ``key = value`` lines that bench.py reads back, together with the
hash of the kernel sources the counters were taken on.
"""
from __future__ import annotations

import argparse
import sqlite3
import sys
from typing import Dict, List, Tuple

FFN_KERNEL = "apk_kernel"
COPY_KERNEL = "__amd_rocclr_copyBuffer"
STREAM_KERNEL = "stream_read"            # libmoe_peaks.so: reads a known number of bytes, writes ~nothing


def _short(name: str) -> str:
    base = name.replace("(anonymous namespace)::", "").replace("void ", "")
    return base.split("(")[0].strip()[:60]


def _dispatches(db: str) -> List[Tuple[str, int, int]]:
    con = sqlite3.connect(db)
    rows = con.execute("select name, dispatch_id, duration from kernels order by start").fetchall()
    con.close()
    return [(n, int(d), int(du)) for n, d, du in rows]


def _pmc(db: str, counter: str) -> List[Tuple[str, int, float]]:
    con = sqlite3.connect(db)
    rows = con.execute("select name, dispatch_id, counter_value from pmc_events where counter_name = ? "
                       "order by dispatch_id", (counter,)).fetchall()
    con.close()
    return [(n, int(d), float(v)) for n, d, v in rows]


def _timed(seq: List, skip: int, take: int) -> List:
    sel = seq[skip:skip + take]
    if len(sel) < take:
        raise SystemExit(f"only {len(seq)} dispatches of the kernel; wanted {skip} + {take}")
    return sel


def stats(args) -> str:
    rows = _dispatches(args.db)
    per: Dict[str, List[int]] = {}
    for n, _, du in rows:
        per.setdefault(n, []).append(du)
    total = sum(sum(v) for v in per.values())
    out = ["# rocprofv3 kernel-trace summary", "", "Command:", "", "```", args.cmd, "```", "",
           "| kernel | calls | total ms | avg us | min us | max us | % |", "|---|---|---|---|---|---|---|"]
    for n, v in sorted(per.items(), key=lambda kv: -sum(kv[1])):
        out.append(f"| {_short(n)} | {len(v)} | {sum(v) / 1e6:.3f} | {sum(v) / len(v) / 1e3:.1f} | "
                   f"{min(v) / 1e3:.1f} | {max(v) / 1e3:.1f} | {100.0 * sum(v) / total:.1f} |")
    ffn = [du for n, _, du in rows if FFN_KERNEL in n and "init" not in n]
    sel = _timed(ffn, args.skip, args.take)
    out += ["", f"{FFN_KERNEL}: all {len(ffn)} dispatches avg {sum(ffn) / len(ffn) / 1e6:.4f} ms; "
            f"timed region (dispatches {args.skip}..{args.skip + args.take - 1}) avg "
            f"{sum(sel) / len(sel) / 1e6:.4f} ms, min {min(sel) / 1e6:.4f}, max {max(sel) / 1e6:.4f}"]
    out += ["", f"timed_avg_ms = {sum(sel) / len(sel) / 1e6:.4f}"]
    return "\n".join(out) + "\n"


def traffic(args) -> str:
    from paper_2607_18002_amd.build import ffn_kernel_hash

    res = {}
    for key, db, counter in (("fetch", args.fetch, "FETCH_SIZE"), ("write", args.write, "WRITE_SIZE")):
        ev = _pmc(db, counter)
        ffn = [v for n, _, v in ev if FFN_KERNEL in n and "init" not in n]
        copy = [v for n, _, v in ev if COPY_KERNEL in n]
        if not copy:
            raise SystemExit(f"{db}: no {COPY_KERNEL} dispatch to calibrate {counter} on")
        big = max(copy)                          # the calibration copy is the largest copy in the run
        cal = [v for v in copy if v >= 0.9 * big]
        kib_copy = sum(cal) / len(cal)
        factor = args.copy_bytes / (kib_copy * 1024.0)
        # the streaming read (same byte count, read only) backs the read-side factor
        stream = [v for n, _, v in ev if STREAM_KERNEL in n]
        kib_stream = sum(stream) / len(stream) if stream else float("nan")
        f_stream = args.copy_bytes / (kib_stream * 1024.0) if stream else float("nan")
        if key == "fetch" and stream:
            factor = f_stream
        sel = _timed(ffn, args.skip, args.take)
        kib = sum(sel) / len(sel)
        res[key] = dict(kib=kib, kib_copy=kib_copy, factor=factor, bytes=kib * 1024.0 * factor, n=len(cal),
                        kib_stream=kib_stream, f_copy=args.copy_bytes / (kib_copy * 1024.0), f_stream=f_stream)
    tot = res["fetch"]["bytes"] + res["write"]["bytes"]
    out = ["# HBM traffic of the persistent FFN kernel (rocprofv3 --pmc)", "",
           f"Workload: {args.workload}", "", "Commands (one counter per run):", "", "```", args.cmd_fetch,
           args.cmd_write, "```", "",
           f"Calibration, in the same runs: a device-to-device copy of {args.copy_bytes:.0f} bytes ({COPY_KERNEL}) "
           f"reads and writes exactly that many bytes, and a streaming read of as many bytes ({STREAM_KERNEL}, "
           "libmoe_peaks.so) reads them and writes one word per workgroup; factor = bytes / (counter KiB * 1024). "
           "FETCH_SIZE takes the streaming read's factor (a read-only kernel of known bytes), WRITE_SIZE the copy's.",
           "", "| counter | kernel KiB/dispatch (timed avg) | copy KiB | copy factor | stream-read KiB | stream factor "
           "| factor used | bytes/launch |", "|---|---|---|---|---|---|---|---|"]
    for key, c in (("fetch", "FETCH_SIZE"), ("write", "WRITE_SIZE")):
        r = res[key]
        fs = f"{r['f_stream']:.4f}" if key == "fetch" else "n/a (writes ~0)"
        out.append(f"| {c} | {r['kib']:.0f} | {r['kib_copy']:.0f} | {r['f_copy']:.4f} | {r['kib_stream']:.0f} | "
                   f"{fs} | {r['factor']:.4f} | {r['bytes']:.4g} |")
    out += ["", f"source_hash = {ffn_kernel_hash()}", f"workload = {args.workload}",
            f"fetch_bytes_per_launch = {res['fetch']['bytes']:.6g}",
            f"write_bytes_per_launch = {res['write']['bytes']:.6g}",
            f"traffic_bytes_per_launch = {tot:.6g}"]
    return "\n".join(out) + "\n"


def counters(args) -> str:
    """Timed-region average per dispatch of each counter in a --pmc database,
    for the persistent kernel and the other kernels of the run."""
    names = args.counters.split(",")
    out = ["# rocprofv3 counters", "", f"Workload: {args.workload}", "", "Command:", "", "```", args.cmd, "```", "",
           "| kernel | dispatches | " + " | ".join(names) + " |", "|---|---|" + "---|" * len(names)]
    vals = {}
    for c in names:
        ev = _pmc(args.db, c)
        # raw block counters come as one row per hardware instance (e.g. 32
        # shader engines): sum them per dispatch
        by_disp: Dict[int, List] = {}
        for n, d, v in ev:
            by_disp.setdefault(d, [n, 0.0])[1] += v
        per: Dict[str, List[float]] = {}
        for d in sorted(by_disp):
            n, v = by_disp[d]
            per.setdefault(_short(n), []).append(v)
        for k, v in per.items():
            if FFN_KERNEL in k and "init" not in k:
                v = _timed(v, args.skip, args.take)
            vals.setdefault(k, {})[c] = (len(v), sum(v) / len(v))
    for k in sorted(vals, key=lambda k: (FFN_KERNEL not in k, k)):
        row = vals[k]
        n = max(x[0] for x in row.values())
        out.append(f"| {k} | {n} | " + " | ".join(f"{row[c][1]:.6g}" if c in row else "" for c in names) + " |")
    ffn = next((vals[k] for k in vals if FFN_KERNEL in k and "init" not in k), None)
    if ffn:
        out += ["", f"source_hash = {__import__('paper_2607_18002_amd.build', fromlist=['x']).ffn_kernel_hash()}"]
        out += [f"{c} = {ffn[c][1]:.6g}" for c in names if c in ffn]
    return "\n".join(out) + "\n"


def main(argv=None) -> int:
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="mode", required=True)
    a = sub.add_parser("stats")
    a.add_argument("db")
    a.add_argument("--skip", type=int, default=0)
    a.add_argument("--take", type=int, default=1)
    a.add_argument("--cmd", default="")
    b = sub.add_parser("traffic")
    b.add_argument("--fetch", required=True)
    b.add_argument("--write", required=True)
    b.add_argument("--skip", type=int, default=0)
    b.add_argument("--take", type=int, default=1)
    b.add_argument("--copy-bytes", type=float, required=True)
    b.add_argument("--workload", required=True)
    b.add_argument("--cmd-fetch", default="")
    b.add_argument("--cmd-write", default="")
    c = sub.add_parser("counters")
    c.add_argument("db")
    c.add_argument("--counters", required=True)
    c.add_argument("--skip", type=int, default=0)
    c.add_argument("--take", type=int, default=1)
    c.add_argument("--workload", default="")
    c.add_argument("--cmd", default="")
    args = ap.parse_args(argv)
    sys.stdout.write({"stats": stats, "traffic": traffic, "counters": counters}[args.mode](args))
    return 0


if __name__ == "__main__":
    sys.exit(main())
