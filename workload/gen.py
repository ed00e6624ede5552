"""Seeded synthetic MoE-layer inputs shaped like the paper's workloads.

The paper evaluates on production models with 256 routed experts and top-8
routing (Evaluation, "Models") and on a single-GPU microbenchmark of
concurrent prefill (8192 tokens) and decode (128 tokens) grouped GEMMs with
decode arriving 10 us after prefill (Evaluation, "Effectiveness of APKs").
Neither the weights nor the request traces exist here, so every input is
drawn from a counter-seeded PCG64 stream:

* seed = SeedSequence([2607, cfg_id, layer, stream, sub])
* stream 0, sub 0       : layer-level draws (expert popularity order, or the
                          router weight of the tiny configuration)
* stream 0, sub 1+2e+m  : expert e's matrix m (m=0 gate/up [2I,H], m=1 down
                          [H,I]); one independent stream per matrix so the
                          32 experts are drawn in parallel threads
* stream 1 / 2          : prefill / decode tokens: logit noise [T,E_g] first,
                          then activations x [T,H]

Values: x ~ N(0,1), W ~ N(0, 0.02), logit noise ~ N(0,1).  Expert skew is a
Zipf popularity bias added to the logits: the expert of popularity rank r
(1 = hottest) gets bias r^-s, so the hottest expert gains one logit.  The
rank order is a seeded permutation with the hottest expert forced onto local
expert 0, so the local share always holds the hot expert.

Storage formats (what the kernels consume): bf16 as uint16 bit patterns
(round to nearest even); fp8 as OCP E4M3FN codes (uint8, max 448, no
infinities) with fp32 scales, one per 128x128 weight block and one per
1x128 activation group, scale = max(amax, 1e-4)/448, codes rounded to
nearest even and saturated at +-448.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, replace
from typing import Optional

import numpy as np

SEED_ROOT = 2607
STREAM_LAYER = 0
STREAM_PREFILL = 1
STREAM_DECODE = 2
E4M3_MAX = 448.0
SCALE_FLOOR = 1e-4
QBLOCK = 128


@dataclass(frozen=True)
class MoEConfig:
    cfg_id: int
    name: str
    E_global: int
    E_local: int
    local_begin: int
    top_k: int
    H: int
    I: int
    prefill_tokens: int
    decode_tokens: int
    n_layers: int
    dtype: str                  # storage type the GPU path computes on: "bf16" | "fp8"
    zipf_s: tuple = ()          # per-layer skew exponent (empty: router logits)
    router: bool = False        # logits = fp32(x @ W_r^T) computed in fp64
    weight_std: float = 0.02


def _cfg4_skews() -> tuple:
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([SEED_ROOT, 4, 99])))
    return tuple(float(v) for v in rng.uniform(0.6, 1.6, size=4))


CONFIGS = {
    1: MoEConfig(1, "tiny-fp32-8e-top2", 8, 8, 0, 2, 256, 512, 48, 16, 1, "bf16", (), True),
    2: MoEConfig(2, "decode-bf16-32of256-top8-h3072-i1536-t512", 256, 32, 0, 8, 3072, 1536,
                 0, 512, 1, "bf16", (1.1,)),
    3: MoEConfig(3, "prefill-bf16-32of256-top8-h3072-i1536-t16384", 256, 32, 0, 8, 3072, 1536,
                 16384, 0, 1, "bf16", (1.1,)),
    4: MoEConfig(4, "mixed-bf16-32of256-top8-h3072-i1536-p8192-d1024-x4layers", 256, 32, 0, 8,
                 3072, 1536, 8192, 1024, 4, "bf16", _cfg4_skews()),
    5: MoEConfig(5, "mixed-fp8-32of256-top8-h6144-i2048-p4096-d1024", 256, 32, 0, 8, 6144, 2048,
                 4096, 1024, 1, "fp8", (1.2,)),
}


def custom_config(base: int = 2, **overrides) -> MoEConfig:
    """A configuration derived from one of CONFIGS with some fields replaced
    (used for small test shapes); give it its own cfg_id so its seeds differ."""
    cfg = replace(CONFIGS[base], **overrides)
    if cfg.zipf_s and len(cfg.zipf_s) < cfg.n_layers:
        cfg = replace(cfg, zipf_s=tuple(cfg.zipf_s[i % len(cfg.zipf_s)] for i in range(cfg.n_layers)))
    return cfg


# --------------------------------------------------------------------------- formats

def bf16_bits(a: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bit patterns (uint16), round to nearest even (finite inputs)."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32).copy()
    r = u >> 16
    r &= 1
    u += r
    u += np.uint32(0x7FFF)
    u >>= 16
    return u.astype(np.uint16)


def e4m3_codes(v: np.ndarray) -> np.ndarray:
    """float32 -> OCP E4M3FN codes (uint8), round to nearest even, saturate at 448."""
    v = np.ascontiguousarray(v, dtype=np.float32)
    a = np.abs(v)
    sign = (np.signbit(v).astype(np.uint8) << 7)
    code = np.zeros(v.shape, dtype=np.uint8)
    small = a < np.float32(2.0 ** -6)
    # subnormal grid: multiples of 2^-9; code == multiple (8 carries into the first normal)
    code[small] = np.rint(a[small] * np.float32(512.0)).astype(np.uint8)
    big = ~small
    u = a[big].view(np.uint32)
    u = (u + (((u >> 20) & 1) + np.uint32(0x7FFFF))) & np.uint32(0xFFF00000)
    sat = u.view(np.float32) > np.float32(E4M3_MAX)
    e = (u >> 23).astype(np.int32) - 127 + 7
    m = ((u >> 20) & 7).astype(np.int32)
    c = (e << 3) | m
    c[sat] = 0x7E
    code[big] = c.astype(np.uint8)
    return code | sign


def _quantize_blocks(w: np.ndarray, bn: int, bk: int):
    """Per-(bn x bk)-block scales and codes for a 2-D float32 matrix."""
    n, k = w.shape
    blocks = w.reshape(n // bn, bn, k // bk, bk)
    amax = np.abs(blocks).max(axis=(1, 3))
    scale = (np.maximum(amax, np.float32(SCALE_FLOOR)) / np.float32(E4M3_MAX)).astype(np.float32)
    q = blocks / scale[:, None, :, None]
    return e4m3_codes(q.reshape(n, k)), scale


# --------------------------------------------------------------------------- draws

def _rng(*key) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([SEED_ROOT, *key])))


def _threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def zipf_bias(cfg: MoEConfig, layer: int) -> np.ndarray:
    """Per-global-expert logit bias rank^-s (float32 [E_global])."""
    s = cfg.zipf_s[layer]
    order = _rng(cfg.cfg_id, layer, STREAM_LAYER, 0).permutation(cfg.E_global)
    hot = int(np.nonzero(order == cfg.local_begin)[0][0])
    order[[0, hot]] = order[[hot, 0]]
    rank = np.empty(cfg.E_global, dtype=np.float64)
    rank[order] = np.arange(1, cfg.E_global + 1, dtype=np.float64)
    return (rank ** (-s)).astype(np.float32)


def _expert_matrix(cfg: MoEConfig, layer: int, e: int, m: int) -> np.ndarray:
    shape = (2 * cfg.I, cfg.H) if m == 0 else (cfg.H, cfg.I)
    w = _rng(cfg.cfg_id, layer, STREAM_LAYER, 1 + 2 * e + m).standard_normal(shape, dtype=np.float32)
    w *= np.float32(cfg.weight_std)
    return w


def make_weights(cfg: MoEConfig, layer: int, keep_f32: bool = False) -> dict:
    """Local expert weights of one layer in the GPU storage format.

    bf16: w_gate_up uint16 [E_l, 2I, H] (gate rows 0..I-1, up rows I..2I-1),
          w_down uint16 [E_l, H, I].
    fp8 : the same shapes as uint8 E4M3FN codes plus fp32 block scales
          w_gate_up_scales [E_l, 2I/128, H/128], w_down_scales [E_l, H/128, I/128].
    keep_f32 adds the drawn float32 matrices (w_gate_up_f32, w_down_f32).
    """
    E, H, I = cfg.E_local, cfg.H, cfg.I
    out = {}
    if cfg.dtype == "bf16":
        out["w_gate_up"] = np.empty((E, 2 * I, H), dtype=np.uint16)
        out["w_down"] = np.empty((E, H, I), dtype=np.uint16)
    else:
        assert H % QBLOCK == 0 and I % QBLOCK == 0, "fp8 needs H and I multiples of 128"
        out["w_gate_up"] = np.empty((E, 2 * I, H), dtype=np.uint8)
        out["w_down"] = np.empty((E, H, I), dtype=np.uint8)
        out["w_gate_up_scales"] = np.empty((E, 2 * I // QBLOCK, H // QBLOCK), dtype=np.float32)
        out["w_down_scales"] = np.empty((E, H // QBLOCK, I // QBLOCK), dtype=np.float32)
    if keep_f32:
        out["w_gate_up_f32"] = np.empty((E, 2 * I, H), dtype=np.float32)
        out["w_down_f32"] = np.empty((E, H, I), dtype=np.float32)

    def job(em):
        e, m = em
        w = _expert_matrix(cfg, layer, e, m)
        name = "w_gate_up" if m == 0 else "w_down"
        if keep_f32:
            out[name + "_f32"][e] = w
        if cfg.dtype == "bf16":
            out[name][e] = bf16_bits(w)
        else:
            codes, scale = _quantize_blocks(w, QBLOCK, QBLOCK)
            out[name][e] = codes
            out[name + "_scales"][e] = scale

    jobs = [(e, m) for e in range(E) for m in range(2)]
    if cfg.H * cfg.I * E >= (1 << 22):
        with ThreadPoolExecutor(_threads()) as ex:
            list(ex.map(job, jobs))
    else:
        for j in jobs:
            job(j)
    if cfg.router:
        out["w_router"] = (_rng(cfg.cfg_id, layer, STREAM_LAYER, 0)
                           .standard_normal((cfg.E_global, H), dtype=np.float32) * np.float32(cfg.weight_std))
    return out


@dataclass
class PhaseInputs:
    phase: str                      # "prefill" | "decode"
    T: int
    logits: np.ndarray              # float32 [T, E_global]
    x: np.ndarray                   # bf16 bits uint16 [T,H] or e4m3 codes uint8 [T,H]
    x_scales: Optional[np.ndarray]  # float32 [T, H/128] for fp8, else None
    x_f32: np.ndarray               # the drawn float32 activations


@dataclass
class LayerInputs:
    cfg: MoEConfig
    layer: int
    weights: dict
    phases: list                    # PhaseInputs, prefill first when present


def make_phase(cfg: MoEConfig, layer: int, phase: str, T: Optional[int] = None,
               w_router: Optional[np.ndarray] = None) -> PhaseInputs:
    stream = STREAM_PREFILL if phase == "prefill" else STREAM_DECODE
    if T is None:
        T = cfg.prefill_tokens if phase == "prefill" else cfg.decode_tokens
    rng = _rng(cfg.cfg_id, layer, stream)
    if cfg.router:
        x = rng.standard_normal((T, cfg.H), dtype=np.float32)
        assert w_router is not None
        logits = (x.astype(np.float64) @ w_router.astype(np.float64).T).astype(np.float32)
    else:
        noise = rng.standard_normal((T, cfg.E_global), dtype=np.float32)
        x = rng.standard_normal((T, cfg.H), dtype=np.float32)
        logits = noise + zipf_bias(cfg, layer)[None, :]
    if cfg.dtype == "bf16":
        return PhaseInputs(phase, T, np.ascontiguousarray(logits), bf16_bits(x), None, x)
    codes, scales = _quantize_blocks(x, 1, QBLOCK)
    return PhaseInputs(phase, T, np.ascontiguousarray(logits), codes, scales, x)


def make_layer(cfg: MoEConfig, layer: int = 0, keep_f32: bool = False) -> LayerInputs:
    w = make_weights(cfg, layer, keep_f32=keep_f32)
    phases = []
    for ph, T in (("prefill", cfg.prefill_tokens), ("decode", cfg.decode_tokens)):
        if T > 0:
            phases.append(make_phase(cfg, layer, ph, T, w.get("w_router")))
    return LayerInputs(cfg, layer, w, phases)
