"""Plain CPU oracle of one GPU's share of a routed-expert MoE layer.

TEST INFRASTRUCTURE ONLY: imported by tests, the smoke check and the
benchmark's CPU-baseline leg, never by the product path.  It shares no code
with the HIP library.  Floating point is evaluated in float64; library
primitives (a stable sort, matrix products, exp) serve as single steps and
nothing is blocked, fused or reordered beyond the definitions below.

What the paper fixes, and the readings taken where it is silent:

* Routing (Background, "MoE LLM Inference"): a router picks a top-k subset of
  the routed experts for each token and the layer output combines the chosen
  experts' outputs.  Reading: softmax gating, top-k on the fp32 logits in
  descending order with ties to the lower expert index, weights renormalised
  over the k selected experts (equal to softmax over all experts, select,
  renormalise).  Experts [local_begin, local_begin+E_local) are this GPU's
  share; other selections get id -1 and keep their weight (no renormalising
  over the local subset: the other expert-parallel ranks hold the rest).
* Permutation ("Prefill-Decode Disaggregation": the contiguous expert layout
  and the masked decode layout; "One-Sided Dispatch and Combine": routing
  fixes each expert's destination and final offset before activations are
  written, into buffers sized for the maximum routed volume).  Reading:
  contiguous -- each expert owns a segment that starts at a multiple of the
  tile height, padding rows zero; masked -- each expert owns a fixed region
  of `slots` rows and a count.  In both, the rows of an expert are its
  assignments a = t*k + j in ascending a.
* Expert FFN (Evaluation, "Implementation": two grouped GEMMs and the
  activation fused into one kernel).  Reading: SwiGLU,
  h = silu(x Wg^T) * (x Wu^T), out = h Wd^T, silu(z) = z / (1 + e^-z), with
  gate rows 0..I-1 and up rows I..2I-1 of the [2I, H] gate/up matrix.
* fp8 path (Evaluation, "Implementation": the fp8 deployment).  Readings:
  OCP E4M3FN codes; activations carry one fp32 scale per row and 128
  columns, weights one per 128 x 128 block; the stored intermediate h is
  re-quantized per row and 128 columns with scale = max(amax, 1e-4) / 448,
  rounding to nearest even and saturating at +-448.  By default the oracle
  keeps h unquantized (the reference the tolerance is stated against); with
  h_fp8 it applies that quantization (quantize_rows).
* Combine (Background, "MoE LLM Inference" and "Large-scale MoE LLM
  Serving"): y[t] = sum over local slots j (ascending) of w[t,j] * out[row].
  A token with no local slot gets exactly zero.
* Footprint, Eq. (3) ("Tile-aware Latency Model"):
  x_moe = sum over experts with m_e > 0 of ceil(m_e / M_t).
* Decode quota, Eq. (4) ("Online SM Reallocation"):
  q' = min(Q_max, ceil_c(q * x_moe / x*_moe)); reading: x*_moe <= 0 means a
  fixed quota (the ratio is taken as 1).
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Optional

import numpy as np

# ----------------------------------------------------------------------------- formats

def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    """bf16 bit patterns (uint16) -> float64: bf16 is the upper half of a float32."""
    u = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return u.view(np.float32).astype(np.float64)


def _e4m3_table() -> np.ndarray:
    """Value of every OCP E4M3FN code: 1 sign, 4 exponent (bias 7), 3 mantissa
    bits; exponent 0 is subnormal (m/8 * 2^-6); S.1111.111 is NaN; no inf."""
    vals = np.empty(256, dtype=np.float64)
    for c in range(256):
        s = -1.0 if c & 0x80 else 1.0
        e = (c >> 3) & 0xF
        m = c & 0x7
        if e == 0xF and m == 0x7:
            vals[c] = np.nan
        elif e == 0:
            vals[c] = s * (m / 8.0) * 2.0 ** -6
        else:
            vals[c] = s * (1.0 + m / 8.0) * 2.0 ** (e - 7)
    return vals


_E4M3 = _e4m3_table()


def e4m3_to_f64(codes: np.ndarray) -> np.ndarray:
    return _E4M3[np.asarray(codes, dtype=np.uint8)]


_E4M3_POS = _E4M3[:0x7F]          # the finite non-negative codes 0x00..0x7E, ascending in value


def e4m3_quantize(v: np.ndarray) -> np.ndarray:
    """float64 -> OCP E4M3FN codes: the nearest representable value, ties to
    the even mantissa, magnitudes beyond 448 saturate to +-448.  Sign from
    the sign bit of the input (so -0.0 gives the negative-zero code)."""
    v = np.asarray(v, dtype=np.float64)
    a = np.minimum(np.abs(v), 448.0)
    hi = np.clip(np.searchsorted(_E4M3_POS, a, side="left"), 0, 0x7E)   # first code with value >= a
    lo = np.maximum(hi - 1, 0)
    d_hi = _E4M3_POS[hi] - a
    d_lo = a - _E4M3_POS[lo]
    pick_lo = (d_lo < d_hi) | ((d_lo == d_hi) & (lo % 2 == 0))
    code = np.where(pick_lo, lo, hi).astype(np.uint8)
    return np.where(np.signbit(v), code | 0x80, code).astype(np.uint8)


def quantize_rows(v: np.ndarray, group: int = 128, floor: float = 1e-4, qmax: float = 448.0):
    """Per-row, per-`group`-column fp8 quantization of the intermediate h
    (reading taken for the paper's fp8 path): scale = max(amax, floor) / qmax,
    code = e4m3(v / scale).  Returns (codes uint8, scales float64)."""
    v = np.asarray(v, dtype=np.float64)
    T, n = v.shape
    g = v.reshape(T, n // group, group)
    scale = np.maximum(np.abs(g).max(axis=2), floor) / qmax
    codes = e4m3_quantize(g / scale[:, :, None]).reshape(T, n)
    return codes, scale


def dequant_rows(x: np.ndarray, x_scales: Optional[np.ndarray] = None, group: int = 128) -> np.ndarray:
    """Activations as float64: bf16 bits, or e4m3 codes times their per-row
    1 x group scale."""
    if x_scales is None:
        return bf16_to_f64(x)
    v = e4m3_to_f64(x)
    T, H = v.shape
    return (v.reshape(T, H // group, group) * np.asarray(x_scales, np.float64)[:, :, None]).reshape(T, H)


def dequant_weight(w: np.ndarray, scales: Optional[np.ndarray] = None, block: int = 128) -> np.ndarray:
    """One expert matrix [N, K] as float64: bf16 bits, or e4m3 codes times the
    scale of their block x block tile."""
    if scales is None:
        return bf16_to_f64(w)
    v = e4m3_to_f64(w)
    N, K = v.shape
    s = np.asarray(scales, np.float64)
    return (v.reshape(N // block, block, K // block, block) * s[:, None, :, None]).reshape(N, K)


# ----------------------------------------------------------------------------- step 1: gating

def route(logits: np.ndarray, top_k: int, local_begin: int, E_local: int):
    """Top-k softmax gating (Background, "MoE LLM Inference").

    Returns (ids int32 [T,k], w float64 [T,k]): ids are local expert ids or -1,
    slots in descending-logit order, ties to the lower global expert index."""
    L = np.asarray(logits, dtype=np.float32).astype(np.float64)
    T, E = L.shape
    if not (1 <= top_k <= E):
        raise ValueError("top_k must be in [1, E_global]")
    if not np.all(np.isfinite(L)):
        raise ValueError("logits must be finite")
    index = np.broadcast_to(np.arange(E), L.shape)
    order = np.lexsort((index, -L), axis=-1)        # primary: logit descending; then index ascending
    sel = order[:, :top_k]
    chosen = np.take_along_axis(L, sel, axis=1)
    m = chosen[:, :1]                                # the largest selected logit
    ex = np.exp(chosen - m)
    w = ex / ex.sum(axis=1, keepdims=True)
    local = sel - local_begin
    ids = np.where((local >= 0) & (local < E_local), local, -1).astype(np.int32)
    return ids, w


# ----------------------------------------------------------------------------- step 2: permutation

@dataclass
class PermuteResult:
    counts: np.ndarray          # int32 [E_local]
    offsets: np.ndarray         # int32 [E_local+1], segment starts, multiples of row_align
    row_to_assign: np.ndarray   # int32 [capacity], -1 on padding / unused rows
    assign_to_row: np.ndarray   # int32 [T*k], -1 for non-local slots
    x_perm: Optional[np.ndarray]  # rows gathered in the input's own storage type, padding rows zero
    x_perm_scales: Optional[np.ndarray] = None  # gathered per-row fp8 group scales, padding rows zero


def permute(ids: np.ndarray, E_local: int, row_align: int, x: Optional[np.ndarray] = None,
            capacity: Optional[int] = None, x_scales: Optional[np.ndarray] = None):
    """Contiguous per-expert layout with final offsets decided after routing."""
    ids = np.asarray(ids, dtype=np.int32)
    T, k = ids.shape
    flat = ids.reshape(-1)
    if np.any(flat >= E_local) or np.any(flat < -1):
        raise ValueError("expert id out of range")
    counts = np.zeros(E_local, dtype=np.int64)
    for e in range(E_local):
        counts[e] = int(np.count_nonzero(flat == e))
    offsets = np.zeros(E_local + 1, dtype=np.int64)
    for e in range(E_local):
        offsets[e + 1] = offsets[e] + -(-counts[e] // row_align) * row_align
    used = int(offsets[-1])
    cap = used if capacity is None else int(capacity)
    if cap < used:
        raise ValueError("capacity too small")
    row_to_assign = np.full(cap, -1, dtype=np.int64)
    assign_to_row = np.full(T * k, -1, dtype=np.int64)
    local_a = np.nonzero(flat >= 0)[0]
    by_expert = local_a[np.argsort(flat[local_a], kind="stable")]   # expert ascending, then a ascending
    fill = offsets[:-1].copy()
    for a in by_expert:
        e = flat[a]
        row_to_assign[fill[e]] = a
        assign_to_row[a] = fill[e]
        fill[e] += 1
    res = PermuteResult(counts.astype(np.int32), offsets.astype(np.int32),
                        row_to_assign.astype(np.int32), assign_to_row.astype(np.int32), None)
    if x is not None:
        x = np.asarray(x)
        xp = np.zeros((cap,) + x.shape[1:], dtype=x.dtype)
        valid = row_to_assign >= 0
        xp[valid] = x[row_to_assign[valid] // k]
        res.x_perm = xp
        if x_scales is not None:
            xs = np.zeros((cap,) + x_scales.shape[1:], dtype=x_scales.dtype)
            xs[valid] = x_scales[row_to_assign[valid] // k]
            res.x_perm_scales = xs
    return res


def permute_masked(ids: np.ndarray, E_local: int, slots: int, x: Optional[np.ndarray] = None,
                   x_scales: Optional[np.ndarray] = None):
    """Masked layout ("Prefill-Decode Disaggregation": the decode layout, one
    fixed region per expert plus a count, no packing pass).  Reading: local
    expert e owns rows [e*slots, (e+1)*slots); its rows are its assignments
    a = t*k + j in ascending a, from the region's start; rows past the count
    hold -1 (and zero activations).  A token selects distinct experts, so a
    region needs at most T rows: slots >= T always suffices."""
    ids = np.asarray(ids, dtype=np.int32)
    T, k = ids.shape
    flat = ids.reshape(-1)
    if np.any(flat >= E_local) or np.any(flat < -1):
        raise ValueError("expert id out of range")
    counts = np.array([np.count_nonzero(flat == e) for e in range(E_local)], dtype=np.int64)
    if np.any(counts > slots):
        raise ValueError("a region holds fewer rows than its expert's assignments")
    offsets = np.arange(E_local + 1, dtype=np.int64) * slots
    cap = E_local * slots
    row_to_assign = np.full(cap, -1, dtype=np.int64)
    assign_to_row = np.full(T * k, -1, dtype=np.int64)
    fill = offsets[:-1].copy()
    for a in range(T * k):                          # ascending a: token, then slot
        e = flat[a]
        if e < 0:
            continue
        row_to_assign[fill[e]] = a
        assign_to_row[a] = fill[e]
        fill[e] += 1
    res = PermuteResult(counts.astype(np.int32), offsets.astype(np.int32),
                        row_to_assign.astype(np.int32), assign_to_row.astype(np.int32), None)
    if x is not None:
        x = np.asarray(x)
        xp = np.zeros((cap,) + x.shape[1:], dtype=x.dtype)
        valid = row_to_assign >= 0
        xp[valid] = x[row_to_assign[valid] // k]
        res.x_perm = xp
        if x_scales is not None:
            xs = np.zeros((cap,) + x_scales.shape[1:], dtype=x_scales.dtype)
            xs[valid] = x_scales[row_to_assign[valid] // k]
            res.x_perm_scales = xs
    return res


# ----------------------------------------------------------------------------- steps 3-5: expert FFN

def expert_hidden(x_rows: np.ndarray, w_gate: np.ndarray, w_up: np.ndarray) -> np.ndarray:
    """GEMM-1 and the activation on float64 rows: h = silu(x Wg^T) * (x Wu^T), [m,I]."""
    g = x_rows @ w_gate.T
    u = x_rows @ w_up.T
    with np.errstate(over="ignore"):
        h = g / (1.0 + np.exp(-g)) * u
    return h


def expert_down(h: np.ndarray, w_down: np.ndarray) -> np.ndarray:
    """GEMM-2 on float64 rows: h [m,I] . Wd^T -> [m,H]."""
    return h @ w_down.T


def expert_ffn(x_rows: np.ndarray, w_gate: np.ndarray, w_up: np.ndarray, w_down: np.ndarray,
               h_fp8: bool = False) -> np.ndarray:
    """SwiGLU expert on float64 rows: x [m,H], Wg/Wu [I,H], Wd [H,I] -> [m,H].
    h_fp8: h passes through the fp8 intermediate format (quantize_rows, then
    dequantized) before the down projection, as the fp8 path stores it."""
    h = expert_hidden(x_rows, w_gate, w_up)
    if h_fp8:
        codes, sc = quantize_rows(h)
        h = dequant_rows(codes, sc)
    return expert_down(h, w_down)


def _expert_weights(weights: dict, e: int, I: int):
    gs = weights.get("w_gate_up_scales")
    ds = weights.get("w_down_scales")
    gu = dequant_weight(weights["w_gate_up"][e], None if gs is None else gs[e])
    wd = dequant_weight(weights["w_down"][e], None if ds is None else ds[e])
    return gu[:I], gu[I:], wd


def grouped_hidden(x_perm_f64: np.ndarray, counts: np.ndarray, offsets: np.ndarray, weights: dict) -> np.ndarray:
    """h of every expert's segment (GEMM-1 and the activation); other rows zero."""
    I = weights["w_down"].shape[2]
    out = np.zeros((x_perm_f64.shape[0], I), dtype=np.float64)
    for e in range(len(counts)):
        m = int(counts[e])
        if m == 0:
            continue
        r0 = int(offsets[e])
        wg, wu, _ = _expert_weights(weights, e, I)
        out[r0:r0 + m] = expert_hidden(x_perm_f64[r0:r0 + m], wg, wu)
    return out


def grouped_down(h_rows: np.ndarray, counts: np.ndarray, offsets: np.ndarray, weights: dict) -> np.ndarray:
    """GEMM-2 of every expert's segment from given h rows; other rows zero."""
    I = weights["w_down"].shape[2]
    out = np.zeros((h_rows.shape[0], weights["w_down"].shape[1]), dtype=np.float64)
    for e in range(len(counts)):
        m = int(counts[e])
        if m == 0:
            continue
        r0 = int(offsets[e])
        _, _, wd = _expert_weights(weights, e, I)
        out[r0:r0 + m] = expert_down(h_rows[r0:r0 + m], wd)
    return out


def grouped_ffn(x_perm_f64: np.ndarray, counts: np.ndarray, offsets: np.ndarray, weights: dict,
                experts: Optional[list] = None, h_fp8: bool = False) -> np.ndarray:
    """Expert FFN over each expert's segment; padding rows and rows of experts
    not listed stay zero.  x_perm_f64 is the dequantized gathered input."""
    E_local = len(counts)
    I = weights["w_down"].shape[2]
    out = np.zeros((x_perm_f64.shape[0], weights["w_down"].shape[1]), dtype=np.float64)
    for e in (range(E_local) if experts is None else experts):
        m = int(counts[e])
        if m == 0:
            continue
        r0 = int(offsets[e])
        wg, wu, wd = _expert_weights(weights, e, I)
        out[r0:r0 + m] = expert_ffn(x_perm_f64[r0:r0 + m], wg, wu, wd, h_fp8)
    return out


# ----------------------------------------------------------------------------- step 6: combine

def combine(y_perm: np.ndarray, assign_to_row: np.ndarray, w: np.ndarray, T: int, top_k: int) -> np.ndarray:
    """y[t] = sum_j w[t,j] * y_perm[assign_to_row[t*k+j]] over local slots, j ascending."""
    H = y_perm.shape[1]
    y = np.zeros((T, H), dtype=np.float64)
    a2r = np.asarray(assign_to_row).reshape(T, top_k)
    for j in range(top_k):
        r = a2r[:, j]
        hit = r >= 0
        y[hit] += w[hit, j][:, None] * y_perm[r[hit]]
    return y


# ----------------------------------------------------------------------------- whole local share

def moe_local_share(logits, x, weights: dict, top_k: int, local_begin: int, E_local: int,
                    row_align: int, x_scales=None, capacity=None, h_fp8: bool = False, slots: int = 0) -> dict:
    """Every step in order; returns all intermediates (float results in float64).
    slots > 0: the masked layout with regions of `slots` rows (row_align and
    capacity are then unused)."""
    ids, w = route(logits, top_k, local_begin, E_local)
    if slots > 0:
        p = permute_masked(ids, E_local, slots, x, x_scales)
    else:
        p = permute(ids, E_local, row_align, x, capacity, x_scales)
    xp = dequant_rows(p.x_perm, p.x_perm_scales)
    y_perm = grouped_ffn(xp, p.counts, p.offsets, weights, h_fp8=h_fp8)
    y = combine(y_perm, p.assign_to_row, w, ids.shape[0], top_k)
    return dict(ids=ids, w=w, perm=p, y_perm=y_perm, y=y)


def token_output(x_row_f64: np.ndarray, ids_row: np.ndarray, w_row: np.ndarray, weights: dict,
                 cache: Optional[dict] = None, h_fp8: bool = False) -> np.ndarray:
    """y for one token, straight from the definition: sum over its local slots
    of w * FFN_e(x).  `cache` may hold dequantized expert weights by id."""
    I = weights["w_down"].shape[2]
    y = np.zeros(weights["w_down"].shape[1], dtype=np.float64)
    for j, e in enumerate(ids_row):
        if e < 0:
            continue
        e = int(e)
        if cache is not None and e in cache:
            wg, wu, wd = cache[e]
        else:
            wg, wu, wd = _expert_weights(weights, e, I)
            if cache is not None:
                cache[e] = (wg, wu, wd)
        y += w_row[j] * expert_ffn(x_row_f64[None, :], wg, wu, wd, h_fp8)[0]
    return y


# ----------------------------------------------------------------------------- scheduling closed forms

def x_moe(counts, M_t: int) -> int:
    """Eq. (3): number of executed row tiles."""
    return int(sum(-(-int(m) // M_t) for m in counts if int(m) > 0))


def count_tiles(counts, M_t: int, n_cols: int, N_t: int) -> int:
    """Tiles of one grouped GEMM with n_cols output columns: x_moe * ceil(n_cols / N_t)."""
    return x_moe(counts, M_t) * (-(-n_cols // N_t))


def decode_quota(q: int, x_moe_now: int, x_moe_star: int, q_max: int, c: int) -> int:
    """Eq. (4) in workgroup units: q' = min(Q_max, ceil_c(q * x_moe / x*_moe)),
    where ceil_c rounds up to a multiple of c.  Integer arithmetic throughout:
    ceil_c(n / d) = c * ceil(n / (d * c)).  A non-positive x*_moe selects the
    fixed quota (the ratio is taken as 1)."""
    if x_moe_star <= 0:
        num, den = int(q), 1
    else:
        num, den = int(q) * int(x_moe_now), int(x_moe_star)
    rounded = c * (-(-num // (den * c)))
    return min(int(q_max), rounded)
