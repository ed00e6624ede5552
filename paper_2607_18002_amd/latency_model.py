"""Tile-aware latency model of the grouped expert FFN (the paper's "Tile-aware
Latency Model", used by its placement search to predict per-rank MoE latency
without profiling every layout).

The paper fits each profiled component with
    t(x, s) = alpha + beta*x + gamma*x*s + delta*x*s^2
and, for the MoE computation, evaluates it at s = 1 with x = x_moe, the
number of row tiles the kernel executes (Eq. 3):
    x_moe = sum over experts e with m_e > 0 of ceil(m_e / M_t),
because a tiled kernel pays one tile's weight transfer and MFMA work per
active expert row tile, however few rows it holds.  At s = 1 the form is the
line t = alpha + beta' * x_moe (beta' = beta + gamma + delta).

This module holds the host arithmetic (footprint, least-squares fits) and a
measurement driver that times the persistent FFN launch on one MI355X over a
sweep of token counts and active experts:

    python -m paper_2607_18002_amd.latency_model [--phase decode|prefill]

prints, per sweep point, tokens, active experts, routed rows, x_moe and the
FFN kernel time, then the fits of time against x_moe and against tokens.
"""
from __future__ import annotations

import argparse
import math
from typing import Dict, List, Sequence, Tuple

import numpy as np


def footprint(counts: Sequence[int], M_t: int) -> int:
    """x_moe of Eq. (3) for per-expert row counts and tile height M_t."""
    if M_t < 1:
        raise ValueError("M_t must be positive")
    return int(sum((int(c) + M_t - 1) // M_t for c in counts if int(c) > 0))


def fit_line(x: Sequence[float], t: Sequence[float]) -> Tuple[float, float, float]:
    """Least-squares t = alpha + beta * x; returns (alpha, beta, r2)."""
    x = np.asarray(x, dtype=np.float64)
    t = np.asarray(t, dtype=np.float64)
    if x.size < 2:
        raise ValueError("need at least two samples")
    A = np.stack([np.ones_like(x), x], axis=1)
    (alpha, beta), *_ = np.linalg.lstsq(A, t, rcond=None)
    pred = alpha + beta * x
    ss_res = float(np.sum((t - pred) ** 2))
    ss_tot = float(np.sum((t - t.mean()) ** 2))
    r2 = 1.0 - ss_res / ss_tot if ss_tot > 0 else 1.0
    return float(alpha), float(beta), r2


def fit_full(x: Sequence[float], s: Sequence[float], t: Sequence[float]) -> Tuple[float, float, float, float]:
    """Least-squares fit of the paper's general form t = a + b x + c x s + d x s^2."""
    x = np.asarray(x, dtype=np.float64)
    s = np.asarray(s, dtype=np.float64)
    t = np.asarray(t, dtype=np.float64)
    A = np.stack([np.ones_like(x), x, x * s, x * s * s], axis=1)
    coef, *_ = np.linalg.lstsq(A, t, rcond=None)
    return tuple(float(c) for c in coef)


def predict(alpha: float, beta: float, x_moe: float) -> float:
    return alpha + beta * x_moe


def routed_logits(T: int, active: int, local_slots: int, E_global: int, E_local: int, top_k: int) -> np.ndarray:
    """Router logits [T, E_global] whose top-k gives every token `local_slots`
    distinct local experts among the first `active` (round robin, so the
    active experts receive near-equal row counts) and fills its other slots
    with distinct non-local experts."""
    if not (1 <= local_slots <= min(active, top_k) and active <= E_local and E_global - E_local >= top_k):
        raise ValueError("inconsistent sweep point")
    L = np.zeros((T, E_global), dtype=np.float32)
    t = np.arange(T)
    for j in range(local_slots):
        L[t, (t * local_slots + j) % active] = 10.0 - 0.01 * j
    span = E_global - E_local
    for j in range(top_k - local_slots):
        L[t, E_local + (t * 7 + j) % span] = 5.0 - 0.01 * j
    return L


def sweep(tokens: Sequence[int], actives: Sequence[int], phase: str = "decode", H: int = 3072, I: int = 1536,
          E_global: int = 256, E_local: int = 32, top_k: int = 8, local_slots: int = 1, reps: int = 10,
          seed: int = 0) -> List[Dict]:
    """Times the persistent FFN launch (one op) at every (tokens, active) point."""
    import torch

    from . import load_library, ops
    from ._lib import MOE_BF16, MOE_DECODE, MOE_PREFILL
    from .pipeline import LayerWeights, MoEPipeline, OpSpec

    load_library()
    dev = torch.device("cuda:0")
    g = torch.Generator(device=dev).manual_seed(seed)
    gu = (torch.randn((E_local, 2 * I, H), generator=g, device=dev) * 0.02).to(torch.bfloat16)
    wd = (torch.randn((E_local, H, I), generator=g, device=dev) * 0.02).to(torch.bfloat16)
    w = LayerWeights(H, I, MOE_BF16, torch.empty_like(gu), torch.empty_like(wd))
    w.load(gu, wd)
    del gu, wd
    ph = MOE_DECODE if phase == "decode" else MOE_PREFILL
    M_t = ops.moe_ffn_tile_shape(ph, MOE_BF16)[0]
    out = []
    for T in tokens:
        x = torch.randn((T, H), generator=g, device=dev).to(torch.bfloat16)
        for act in actives:
            ls = min(local_slots, act)
            logits = torch.from_numpy(routed_logits(T, act, ls, E_global, E_local, top_k)).to(dev)
            spec = OpSpec(phase=ph, layer=0, logits=logits, x=x, weights=w, E_local=E_local, top_k=top_k,
                          local_begin=0)
            pipe = MoEPipeline([spec], fused_gather=True)
            pipe.route()
            pipe.permute()
            for _ in range(3):
                pipe.ffn()
            torch.cuda.synchronize()
            if pipe.statuses() != (0, 0):
                raise RuntimeError(f"device status {pipe.statuses()} at T={T} active={act}")
            ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
            for a, b in ev:
                a.record()
                pipe.ffn()
                b.record()
            torch.cuda.synchronize()
            ms = float(np.median([a.elapsed_time(b) for a, b in ev]))
            counts = pipe.bufs[0].counts.cpu().numpy()
            out.append(dict(tokens=T, active=int((counts > 0).sum()), rows=int(counts.sum()),
                            x_moe=footprint(counts, M_t), ms=ms))
            del pipe
    return out


def main(argv=None) -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--phase", choices=("decode", "prefill"), default="decode")
    ap.add_argument("--tokens", default="16,64,256,1024,4096")
    ap.add_argument("--actives", default="1,2,4,8,16,32")
    args = ap.parse_args(argv)
    pts = sweep([int(v) for v in args.tokens.split(",")], [int(v) for v in args.actives.split(",")], args.phase)
    print("| tokens | active experts | routed rows | x_moe | FFN kernel ms |")
    print("|---|---|---|---|---|")
    for p in pts:
        print(f"| {p['tokens']} | {p['active']} | {p['rows']} | {p['x_moe']} | {p['ms']:.4f} |")
    a, b, r2 = fit_line([p["x_moe"] for p in pts], [p["ms"] for p in pts])
    a2, b2, r2t = fit_line([p["tokens"] for p in pts], [p["ms"] for p in pts])
    a3, b3, r2r = fit_line([p["rows"] for p in pts], [p["ms"] for p in pts])
    print(f"\nfit on x_moe : t = {a * 1e3:.1f} us + {b * 1e3:.2f} us * x_moe   (R^2 = {r2:.4f})")
    print(f"fit on tokens: t = {a2 * 1e3:.1f} us + {b2 * 1e6:.2f} ns * tokens (R^2 = {r2t:.4f})")
    print(f"fit on rows  : t = {a3 * 1e3:.1f} us + {b3 * 1e6:.2f} ns * rows   (R^2 = {r2r:.4f})")
    err = [abs(predict(a, b, p["x_moe"]) - p["ms"]) / p["ms"] for p in pts]
    print(f"x_moe fit: max relative error {max(err) * 100:.1f}%, mean {np.mean(err) * 100:.1f}%")
    return 0


if __name__ == "__main__":
    raise SystemExit(main())
