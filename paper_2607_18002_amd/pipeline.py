"""Buffer plumbing around the four C-ABI calls for a set of MoE operations
(layers x phases) that share one persistent FFN launch.  Allocates the
capacity-sized buffers once (device memory comes from torch), then issues
route -> permute for every op (one batched launch per pass), one
moe_grouped_ffn_persistent over all ops, and one batched combine, all on one
stream.  No arithmetic happens here."""
from __future__ import annotations

import ctypes as C
from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np
import torch

from . import ops as K
from ._lib import (MOE_BF16, MOE_DECODE, MOE_F32, MOE_FP8_E4M3, MOE_LAYOUT_PACKED, MOE_PREFILL, OpDesc, OpStats, SchedConfig,
                   TraceRec)

TRACE_DTYPE = np.dtype([("op", "<i2"), ("stage", "<i2"), ("wg", "<i2"), ("xcc", "<i2"), ("expert", "<i4"),
                        ("mblk", "<i4"), ("nblk", "<i2"), ("rows", "<i2"), ("quota_seen", "<i2"),
                        ("phases_seen", "u1"), ("how", "u1"), ("t_boundary", "<u8"),
                        ("t_polled", "<u8"), ("t_claim", "<u8"), ("t_start", "<u8"), ("t_end", "<u8"),
                        ("c_start", "<u8"), ("c_end", "<u8")])
STATS_DTYPE = np.dtype([("t_seen", "<u8"), ("t_ready", "<u8"), ("t_first", "<u8"), ("t_done", "<u8"), ("x_moe", "<i4"),
                        ("n_tiles", "<i4"), ("quota", "<i4"), ("reserved", "<i4")])
assert TRACE_DTYPE.itemsize == C.sizeof(TraceRec) and STATS_DTYPE.itemsize == C.sizeof(OpStats)


def split_trace(recs: np.ndarray, n_wg: int) -> np.ndarray:
    """The records of a trace buffer's per-workgroup blocks, each block taken up
    to its terminator (op = -1) or its end, in order of tile start."""
    per = len(recs) // n_wg
    out = []
    for w in range(n_wg):
        blk = recs[w * per:(w + 1) * per]
        end = np.nonzero(blk["op"] < 0)[0]
        out.append(blk[: end[0] if len(end) else per])
    allr = np.concatenate(out) if out else recs[:0]
    return allr[np.argsort(allr["t_start"], kind="stable")]


def bf16_tensor(bits: np.ndarray, device) -> torch.Tensor:
    """bf16 bit patterns (uint16 numpy) -> device bf16 tensor (same bits)."""
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).to(device)


def bits_of(t: torch.Tensor) -> np.ndarray:
    """device bf16 tensor -> uint16 numpy bit patterns."""
    return t.detach().view(torch.int16).cpu().numpy().view(np.uint16)


@dataclass
class LayerWeights:
    """Expert weights of one layer on the device, in the FFN kernel's packed
    layout (moe_pack_weights); load() converts row-major [E, N, K] tensors."""
    H: int
    I: int
    dtype: int                                  # MOE_BF16 | MOE_FP8_E4M3
    w_gate_up: torch.Tensor                     # packed [E_l, 2I, H]
    w_down: torch.Tensor                        # packed [E_l, H, I]
    w_gate_up_scales: Optional[torch.Tensor] = None
    w_down_scales: Optional[torch.Tensor] = None
    layout: int = MOE_LAYOUT_PACKED

    def load(self, w_gate_up: torch.Tensor, w_down: torch.Tensor) -> None:
        """Overwrite with new row-major device weights (packed on the device)."""
        K.moe_pack_weights(w_gate_up, self.w_gate_up)
        K.moe_pack_weights(w_down, self.w_down)

    @staticmethod
    def from_numpy(w: dict, H: int, I: int, device) -> "LayerWeights":
        if w["w_gate_up"].dtype == np.uint16:
            gu, wd = bf16_tensor(w["w_gate_up"], device), bf16_tensor(w["w_down"], device)
            lw = LayerWeights(H, I, MOE_BF16, torch.empty_like(gu), torch.empty_like(wd))
            lw.load(gu, wd)
            del gu, wd
            return lw
        gu, wd = torch.from_numpy(w["w_gate_up"]).to(device), torch.from_numpy(w["w_down"]).to(device)
        lw = LayerWeights(H, I, MOE_FP8_E4M3, torch.empty_like(gu), torch.empty_like(wd),
                          torch.from_numpy(np.ascontiguousarray(w["w_gate_up_scales"], dtype=np.float32)).to(device),
                          torch.from_numpy(np.ascontiguousarray(w["w_down_scales"], dtype=np.float32)).to(device))
        lw.load(gu, wd)
        del gu, wd
        return lw


@dataclass
class OpSpec:
    phase: int
    layer: int
    logits: torch.Tensor                        # [T, E_global] f32, device
    x: torch.Tensor                             # [T, H] bf16 or uint8 codes, device
    weights: LayerWeights
    E_local: int
    top_k: int
    local_begin: int = 0
    x_scales: Optional[torch.Tensor] = None     # [T, H/128] f32 (fp8)
    release_after_ns: int = -1
    depends_on_op: int = -1
    gap_ns: int = 0
    release_word: Optional[torch.Tensor] = None  # uint32 tensor (device or pinned host)


@dataclass
class OpBuffers:
    spec: OpSpec
    T: int
    capacity: int
    row_align: int
    topk_ids: torch.Tensor
    topk_w: torch.Tensor
    counts: torch.Tensor
    offsets: torch.Tensor
    row_to_assign: torch.Tensor
    assign_to_row: torch.Tensor
    x_perm: Optional[torch.Tensor]              # None when the FFN gathers x rows itself
    x_perm_scales: Optional[torch.Tensor]
    h: torch.Tensor
    h_scales: Optional[torch.Tensor]
    y_perm: torch.Tensor
    y: torch.Tensor
    perm_ws: torch.Tensor
    done_word: torch.Tensor
    slots: int = 0                              # masked layout: rows per local expert (0: contiguous layout)
    place_ws: Optional[torch.Tensor] = None     # masked layout: the routing launch's placement workspace


class MoEPipeline:
    def __init__(self, specs: List[OpSpec], n_workgroups: int = 0, decode_quota_wg: int = 64,
                 decode_quota_max_wg: int = 0, x_moe_expected: int = 0, round_multiple: int = 8,
                 trace_capacity: int = 0, spin_limit: int = 0, abort_word: Optional[torch.Tensor] = None,
                 y_dtype: torch.dtype = torch.bfloat16, fused_gather: bool = False, group_row_tiles: int = 0,
                 static_partition: bool = False, fused_combine: bool = False, masked_decode: bool = False,
                 prefill_tile_rows: int = 0,
                 masked_prefill: bool = False):
        """fused_gather: GEMM-1 reads its rows straight from x through row_to_assign
        (permute then only builds the maps), instead of from a permuted copy x_perm.
        fused_combine: the persistent kernel writes y itself (combine tiles after
        each op's GEMM tiles), and combine() launches nothing.
        masked_decode / masked_prefill: ops of that phase use the masked layout
        (a region of slots rows per local expert, placed by the routing launch;
        permute() skips them)."""
        if not specs:
            raise ValueError("no operations")
        self.device = specs[0].logits.device
        self.fused_gather = fused_gather
        self.fused_combine = fused_combine
        if (masked_decode or masked_prefill) and not fused_gather:
            raise ValueError("the masked layout needs fused_gather (nothing copies rows into x_perm)")
        dev = self.device
        self.bufs: List[OpBuffers] = []
        for s in specs:
            T = s.logits.shape[0]
            H, I = s.weights.H, s.weights.I
            fp8 = s.weights.dtype == MOE_FP8_E4M3
            ra = K.moe_ffn_row_align(s.phase, s.weights.dtype)
            if ra <= 0:
                raise ValueError(f"no FFN tile class for phase={s.phase} dtype={s.weights.dtype}")
            masked = (masked_decode if s.phase == MOE_DECODE else masked_prefill) and T > 0
            slots = (T + 31) // 32 * 32 if masked else 0
            cap = s.E_local * slots if masked else T * min(s.top_k, s.E_local) + s.E_local * (ra - 1)
            act = torch.uint8 if fp8 else torch.bfloat16
            self.bufs.append(OpBuffers(
                spec=s, T=T, capacity=cap, row_align=ra,
                topk_ids=torch.empty((T, s.top_k), dtype=torch.int32, device=dev),
                topk_w=torch.empty((T, s.top_k), dtype=torch.float32, device=dev),
                counts=torch.zeros(s.E_local, dtype=torch.int32, device=dev),
                offsets=(torch.arange(s.E_local + 1, dtype=torch.int32, device=dev) * slots if masked
                         else torch.zeros(s.E_local + 1, dtype=torch.int32, device=dev)),
                row_to_assign=torch.full((cap,), -1, dtype=torch.int32, device=dev),
                assign_to_row=torch.empty((T * s.top_k,), dtype=torch.int32, device=dev),
                x_perm=None if fused_gather else torch.zeros((cap, H), dtype=act, device=dev),
                x_perm_scales=(torch.zeros((cap, H // 128), dtype=torch.float32, device=dev)
                               if fp8 and not fused_gather else None),
                h=torch.zeros((cap, I), dtype=act, device=dev),
                h_scales=torch.zeros((cap, I // 128), dtype=torch.float32, device=dev) if fp8 else None,
                y_perm=torch.zeros((cap, H), dtype=torch.bfloat16, device=dev),
                y=torch.empty((T, H), dtype=y_dtype, device=dev),
                perm_ws=torch.zeros((max(1, K.moe_permute_workspace_bytes(T, s.top_k, s.E_local)),),
                                    dtype=torch.uint8, device=dev),
                done_word=torch.zeros(1, dtype=torch.int32, device=dev),
                slots=slots,
                place_ws=(torch.zeros((K.moe_route_place_workspace_bytes(T, s.E_local),), dtype=torch.uint8,
                                      device=dev) if masked else None),
            ))
        self.error_flag = torch.zeros(1, dtype=torch.int32, device=dev)
        self.status = torch.zeros(1, dtype=torch.int32, device=dev)
        self.trace_capacity = trace_capacity
        self.trace = torch.zeros((max(1, trace_capacity) * TRACE_DTYPE.itemsize,), dtype=torch.uint8, device=dev)
        self.stats = torch.zeros((len(specs) * STATS_DTYPE.itemsize,), dtype=torch.uint8, device=dev)
        self.abort_word = abort_word
        self.cfg = SchedConfig(n_workgroups=n_workgroups, decode_quota_wg=decode_quota_wg,
                               decode_quota_max_wg=decode_quota_max_wg, x_moe_expected=x_moe_expected,
                               round_multiple=round_multiple, group_row_tiles=group_row_tiles,
                               abort_word=abort_word.data_ptr() if abort_word is not None else None,
                               trace=self.trace.data_ptr() if trace_capacity > 0 else None,
                               trace_capacity=trace_capacity, op_stats=self.stats.data_ptr(),
                               spin_limit=spin_limit, static_partition=int(static_partition),
                               prefill_tile_rows=prefill_tile_rows)
        self._descs = [self._desc(i, b, fused_gather, fused_combine) for i, b in enumerate(self.bufs)]
        self._route_args = []
        for b in self.bufs:
            s = b.spec
            if b.place_ws is None:
                self._route_args.append(K.route_args(s.logits, s.top_k, s.local_begin, s.E_local, b.topk_ids,
                                                     b.topk_w))
            else:
                self._route_args.append(K.route_args(s.logits, s.top_k, s.local_begin, s.E_local, b.topk_ids,
                                                     b.topk_w, slots=b.slots, counts=b.counts, place_ws=b.place_ws,
                                                     assign_to_row=b.assign_to_row, row_to_assign=b.row_to_assign,
                                                     error_flag=self.error_flag))
        self._permute_args = [K.permute_args(b.topk_ids, b.spec.E_local, b.spec.x, b.spec.x_scales, b.row_align,
                                             b.capacity, b.counts, b.offsets, b.row_to_assign, b.assign_to_row,
                                             b.x_perm, b.x_perm_scales, b.perm_ws, self.error_flag)
                              for b in self.bufs if b.place_ws is None]
        self._combine_args = [K.combine_args(b.y_perm, b.assign_to_row, b.topk_w, b.T, b.spec.top_k, b.y)
                              for b in self.bufs]
        self.ffn_ws = torch.zeros((K.moe_ffn_workspace_bytes(self.descs, self.cfg),), dtype=torch.uint8, device=dev)

    @staticmethod
    def _desc(i: int, b: OpBuffers, fused_gather: bool = False, fused_combine: bool = False) -> OpDesc:
        s, w = b.spec, b.spec.weights
        p = lambda t: None if t is None else t.data_ptr()  # noqa: E731
        gathered = {}
        if fused_gather:
            gathered = dict(x=p(s.x), x_scales=p(s.x_scales), row_to_assign=p(b.row_to_assign), T=b.T,
                            top_k=s.top_k)
        if fused_combine:
            gathered.update(T=b.T, top_k=s.top_k, assign_to_row=p(b.assign_to_row), topk_w=p(b.topk_w), y=p(b.y),
                            y_dtype=MOE_F32 if b.y.dtype == torch.float32 else MOE_BF16)
        return OpDesc(**gathered, phase=s.phase, layer=s.layer, E_local=s.E_local, H=w.H, I=w.I, capacity=b.capacity,
                      row_align=b.row_align, dtype=w.dtype, counts=p(b.counts), offsets=p(b.offsets),
                      x_perm=p(b.x_perm), x_perm_scales=p(b.x_perm_scales), w_gate_up=p(w.w_gate_up),
                      w_gate_up_scales=p(w.w_gate_up_scales), w_down=p(w.w_down),
                      w_down_scales=p(w.w_down_scales), h=p(b.h), h_scales=p(b.h_scales), y_perm=p(b.y_perm),
                      release_word=p(s.release_word), release_after_ns=s.release_after_ns,
                      depends_on_op=s.depends_on_op, weight_layout=w.layout, gap_ns=s.gap_ns,
                      done_word=p(b.done_word))

    # ---------------------------------------------------------------- the four calls
    # Every op's route, permute and combine go out as one launch per pass
    # (moe_*_batch); batched=False issues the per-op calls instead.
    @property
    def descs(self):
        return self._descs

    def route(self, stream=None, batched: bool = True):
        if batched:
            K.moe_topk_route_batch(self._route_args, stream)
            return
        if any(b.place_ws is not None for b in self.bufs):
            raise ValueError("masked ops are routed by the batched call only")
        for b in self.bufs:
            s = b.spec
            K.moe_topk_route(s.logits, s.top_k, s.local_begin, s.E_local, b.topk_ids, b.topk_w, stream)

    def permute(self, stream=None, batched: bool = True):
        if batched:
            if self._permute_args:
                K.moe_permute_batch(self._permute_args, stream)
            return
        for b in self.bufs:
            if b.place_ws is not None:              # masked: routing placed the rows
                continue
            s = b.spec
            K.moe_permute(b.topk_ids, s.E_local, s.x, s.x_scales, b.row_align, b.capacity, b.counts, b.offsets,
                          b.row_to_assign, b.assign_to_row, b.x_perm, b.x_perm_scales, b.perm_ws,
                          self.error_flag, stream)

    def ffn(self, stream=None):
        K.moe_grouped_ffn_persistent(self.descs, self.cfg, self.ffn_ws, self.status, stream)

    def ffn_plain(self, stream=None):
        """The comparison baseline: the same tiles as plain grids, op after op."""
        K.moe_grouped_ffn_plain(self.descs, self.ffn_ws, self.status, stream)

    def combine(self, stream=None, batched: bool = True):
        if self.fused_combine:                     # the persistent kernel wrote y
            return
        if batched:
            K.moe_combine_batch(self._combine_args, stream)
            return
        for b in self.bufs:
            K.moe_combine(b.y_perm, b.assign_to_row, b.topk_w, b.T, b.spec.top_k, b.y, stream=stream)

    def run(self, stream=None):
        self.route(stream)
        self.permute(stream)
        self.ffn(stream)
        self.combine(stream)

    # ---------------------------------------------------------------- read-back helpers
    def statuses(self):
        return int(self.error_flag.item()), int(self.status.item())

    def trace_records(self) -> np.ndarray:
        """The last launch's tile records: workgroup w wrote its tiles in order
        into block w of trace_capacity // n_wg records, ended by a record with
        op = -1 unless the block is full."""
        n_wg = int(self.ffn_ws[16:20].view(torch.int32).item())
        if self.trace_capacity <= 0 or n_wg <= 0:
            return np.zeros(0, dtype=TRACE_DTYPE)
        return split_trace(self.trace.cpu().numpy().view(TRACE_DTYPE), n_wg)

    def kernel_t0(self) -> int:
        """Device wall-clock tick at which the last persistent launch started."""
        return int(self.ffn_ws[:8].view(torch.int64).item())

    def launch_ticks(self):
        """(init kernel done, first workgroup entry, last workgroup exit) of the
        last launch, in device wall-clock ticks."""
        h = self.ffn_ws[:40].view(torch.int64).cpu().numpy()
        return int(h[3]), int(h[0]), int(h[4])

    def op_stats(self) -> np.ndarray:
        return self.stats.cpu().numpy().view(STATS_DTYPE)
