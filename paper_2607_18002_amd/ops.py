"""Thin Python binding of the C ABI (include/moe_apk.h): same names, torch
tensors in, device pointers and the current HIP stream out.  Every step runs
in the HIP library; nothing here computes."""
from __future__ import annotations

import ctypes as C
from typing import Optional, Sequence

import torch

from . import _lib
from ._lib import (MOE_BF16, MOE_F32, MOE_FP8_E4M3, CombineArgs, OpDesc, PermuteArgs, RouteArgs, SchedConfig, check,
                   load_library)


def _stream(stream: Optional[torch.cuda.Stream]) -> int:
    s = stream if stream is not None else torch.cuda.current_stream()
    return int(s.cuda_stream)


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("expected a device tensor")
    if not t.is_contiguous():
        raise ValueError("expected a contiguous tensor")
    return t.data_ptr()


def act_dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return MOE_BF16
    if t.dtype in (torch.uint8, getattr(torch, "float8_e4m3fn", torch.uint8)):
        return MOE_FP8_E4M3
    raise ValueError(f"unsupported activation dtype {t.dtype}")


def moe_topk_route(logits: torch.Tensor, top_k: int, local_begin: int, E_local: int,
                   topk_ids: Optional[torch.Tensor] = None, topk_w: Optional[torch.Tensor] = None,
                   stream=None):
    lib = load_library()
    T, E = logits.shape
    if topk_ids is None:
        topk_ids = torch.empty((T, top_k), dtype=torch.int32, device=logits.device)
    if topk_w is None:
        topk_w = torch.empty((T, top_k), dtype=torch.float32, device=logits.device)
    check(lib.moe_topk_route(_ptr(logits), T, E, top_k, local_begin, E_local, _ptr(topk_ids), _ptr(topk_w),
                             _stream(stream)), "moe_topk_route")
    return topk_ids, topk_w


def _array(cls, entries):
    arr = (cls * len(entries))()
    for i, e in enumerate(entries):
        arr[i] = e
    return arr


def moe_topk_route_batch(entries: Sequence[RouteArgs], stream=None) -> None:
    """moe_topk_route for several ops in one launch (entries: RouteArgs)."""
    check(load_library().moe_topk_route_batch(_array(RouteArgs, entries), len(entries), _stream(stream)),
          "moe_topk_route_batch")


def route_args(logits: torch.Tensor, top_k: int, local_begin: int, E_local: int, topk_ids: torch.Tensor,
               topk_w: torch.Tensor, slots: int = 0, counts: Optional[torch.Tensor] = None,
               place_ws: Optional[torch.Tensor] = None, assign_to_row: Optional[torch.Tensor] = None,
               row_to_assign: Optional[torch.Tensor] = None, error_flag: Optional[torch.Tensor] = None) -> RouteArgs:
    """One entry of moe_topk_route_batch; with counts given it also places the
    local slots in the masked layout (slots rows per local expert)."""
    T, E = logits.shape
    return RouteArgs(logits=_ptr(logits), T=T, E_global=E, top_k=top_k, local_begin=local_begin, E_local=E_local,
                     topk_ids=_ptr(topk_ids), topk_w=_ptr(topk_w), slots=slots, counts=_ptr(counts),
                     place_ws=_ptr(place_ws), assign_to_row=_ptr(assign_to_row), row_to_assign=_ptr(row_to_assign),
                     error_flag=_ptr(error_flag))


def moe_route_place_workspace_bytes(T: int, E_local: int) -> int:
    return int(load_library().moe_route_place_workspace_bytes(T, E_local))


def moe_permute_workspace_bytes(T: int, top_k: int, E_local: int) -> int:
    return int(load_library().moe_permute_workspace_bytes(T, top_k, E_local))


def moe_permute(topk_ids: torch.Tensor, E_local: int, x: torch.Tensor, x_scales: Optional[torch.Tensor],
                row_align: int, capacity: int, counts: torch.Tensor, offsets: torch.Tensor,
                row_to_assign: torch.Tensor, assign_to_row: torch.Tensor, x_perm: Optional[torch.Tensor],
                x_perm_scales: Optional[torch.Tensor], workspace: torch.Tensor, error_flag: torch.Tensor,
                stream=None) -> None:
    lib = load_library()
    T, k = topk_ids.shape
    H = x.shape[1]
    check(lib.moe_permute(_ptr(topk_ids), T, k, E_local, _ptr(x), act_dtype_code(x), _ptr(x_scales), H,
                          row_align, capacity, _ptr(counts), _ptr(offsets), _ptr(row_to_assign),
                          _ptr(assign_to_row), _ptr(x_perm), _ptr(x_perm_scales), _ptr(workspace),
                          _ptr(error_flag), _stream(stream)), "moe_permute")


def permute_args(topk_ids: torch.Tensor, E_local: int, x: torch.Tensor, x_scales: Optional[torch.Tensor],
                 row_align: int, capacity: int, counts: torch.Tensor, offsets: torch.Tensor,
                 row_to_assign: torch.Tensor, assign_to_row: torch.Tensor, x_perm: Optional[torch.Tensor],
                 x_perm_scales: Optional[torch.Tensor], workspace: torch.Tensor,
                 error_flag: torch.Tensor) -> PermuteArgs:
    T, k = topk_ids.shape
    return PermuteArgs(topk_ids=_ptr(topk_ids), T=T, top_k=k, E_local=E_local, x_dtype=act_dtype_code(x),
                       x=_ptr(x), x_scales=_ptr(x_scales), H=x.shape[1], row_align=row_align, capacity=capacity,
                       counts=_ptr(counts), offsets=_ptr(offsets), row_to_assign=_ptr(row_to_assign),
                       assign_to_row=_ptr(assign_to_row), x_perm=_ptr(x_perm), x_perm_scales=_ptr(x_perm_scales),
                       workspace=_ptr(workspace), error_flag=_ptr(error_flag))


def moe_permute_batch(entries: Sequence[PermuteArgs], stream=None) -> None:
    """moe_permute for several ops, one launch per pass (entries: PermuteArgs)."""
    check(load_library().moe_permute_batch(_array(PermuteArgs, entries), len(entries), _stream(stream)),
          "moe_permute_batch")


def moe_ffn_row_align(phase: int, dtype: int) -> int:
    return int(load_library().moe_ffn_row_align(phase, dtype))


def moe_ffn_tile_shape(phase: int, dtype: int):
    """(rows, columns, K step) of the FFN output tile for ops of this phase and dtype."""
    bm, bn, bk = C.c_int32(), C.c_int32(), C.c_int32()
    check(load_library().moe_ffn_tile_shape(phase, dtype, C.byref(bm), C.byref(bn), C.byref(bk)),
          "moe_ffn_tile_shape")
    return bm.value, bn.value, bk.value


def _op_array(ops: Sequence[OpDesc]):
    arr = (OpDesc * len(ops))()
    for i, o in enumerate(ops):
        arr[i] = o
    return arr


def moe_ffn_workspace_bytes(ops: Sequence[OpDesc], cfg: SchedConfig) -> int:
    lib = load_library()
    return int(lib.moe_ffn_workspace_bytes(_op_array(ops), len(ops), C.byref(cfg)))


def moe_grouped_ffn_persistent(ops: Sequence[OpDesc], cfg: SchedConfig, workspace: torch.Tensor,
                               status_word: torch.Tensor, stream=None) -> None:
    lib = load_library()
    check(lib.moe_grouped_ffn_persistent(_op_array(ops), len(ops), C.byref(cfg), _ptr(workspace),
                                         _ptr(status_word), _stream(stream)), "moe_grouped_ffn_persistent")


def moe_grouped_ffn_persistent_noalloc(ops: Sequence[OpDesc], cfg: SchedConfig, status_word: torch.Tensor,
                                       stream=None) -> None:
    """The persistent FFN launch with the library's static scheduler workspace."""
    lib = load_library()
    check(lib.moe_grouped_ffn_persistent_noalloc(_op_array(ops), len(ops), C.byref(cfg), _ptr(status_word),
                                                 _stream(stream)), "moe_grouped_ffn_persistent_noalloc")


def moe_grouped_ffn_plain(ops: Sequence[OpDesc], workspace: torch.Tensor, status_word: torch.Tensor,
                          stream=None) -> None:
    """The same tiles as plain grids per op (planning, GEMM-1, GEMM-2 launches): a baseline."""
    lib = load_library()
    check(lib.moe_grouped_ffn_plain(_op_array(ops), len(ops), _ptr(workspace), _ptr(status_word), _stream(stream)),
          "moe_grouped_ffn_plain")


def moe_combine(y_perm: torch.Tensor, assign_to_row: torch.Tensor, topk_w: torch.Tensor, T: int, top_k: int,
                y: Optional[torch.Tensor] = None, out_dtype: torch.dtype = torch.bfloat16, stream=None):
    lib = load_library()
    H = y_perm.shape[1]
    if y is None:
        y = torch.empty((T, H), dtype=out_dtype, device=y_perm.device)
    code = MOE_BF16 if y.dtype == torch.bfloat16 else MOE_F32 if y.dtype == torch.float32 else None
    if code is None:
        raise ValueError("y must be bf16 or f32")
    check(lib.moe_combine(_ptr(y_perm), _ptr(assign_to_row), _ptr(topk_w), T, top_k, H, _ptr(y), code,
                          _stream(stream)), "moe_combine")
    return y


def combine_args(y_perm: torch.Tensor, assign_to_row: torch.Tensor, topk_w: torch.Tensor, T: int, top_k: int,
                 y: torch.Tensor) -> CombineArgs:
    code = MOE_BF16 if y.dtype == torch.bfloat16 else MOE_F32 if y.dtype == torch.float32 else None
    if code is None:
        raise ValueError("y must be bf16 or f32")
    return CombineArgs(y_perm=_ptr(y_perm), assign_to_row=_ptr(assign_to_row), topk_w=_ptr(topk_w), T=T,
                       top_k=top_k, H=y_perm.shape[1], y_dtype=code, y=_ptr(y))


def moe_combine_batch(entries: Sequence[CombineArgs], stream=None) -> None:
    """moe_combine for several ops in one launch (entries: CombineArgs)."""
    check(load_library().moe_combine_batch(_array(CombineArgs, entries), len(entries), _stream(stream)),
          "moe_combine_batch")


def moe_pack_weights(src: torch.Tensor, dst: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """[E, N, K] bf16 or fp8-code (uint8) row-major -> the FFN kernel's packed
    weight layout (same shape and size)."""
    lib = load_library()
    E, N, K = src.shape
    if dst is None:
        dst = torch.empty_like(src)
    check(lib.moe_pack_weights(_ptr(src), _ptr(dst), E, N, K, act_dtype_code(src), _stream(stream)),
          "moe_pack_weights")
    return dst


def moe_x_moe(counts: Sequence[int], M_t: int) -> int:
    lib = load_library()
    arr = (C.c_int32 * len(counts))(*[int(c) for c in counts])
    return int(lib.moe_x_moe(arr, len(counts), M_t))


def moe_decode_quota(q: int, x_moe: int, x_moe_expected: int, q_max: int, round_multiple: int) -> int:
    return int(load_library().moe_decode_quota(q, x_moe, x_moe_expected, q_max, round_multiple))


def status_string(status: int) -> str:
    return load_library().moe_status_string(status).decode()


__all__ = ["moe_topk_route", "moe_topk_route_batch", "moe_route_place_workspace_bytes", "moe_permute_workspace_bytes", "moe_permute", "moe_permute_batch",
           "moe_ffn_row_align", "moe_ffn_tile_shape", "moe_ffn_workspace_bytes", "moe_grouped_ffn_persistent",
           "moe_grouped_ffn_persistent_noalloc", "moe_grouped_ffn_plain", "moe_combine", "moe_combine_batch", "moe_pack_weights", "moe_x_moe", "moe_decode_quota", "status_string",
           "route_args", "permute_args", "combine_args", "OpDesc", "SchedConfig", "_lib"]


def moe_sched_layout(counts, offsets, M_t: int, gmax: int, n1: int, n2: int):
    """The tile layout the persistent kernel builds for one op (host-side, the
    kernel's own index arithmetic): (row_tiles [x_moe,4], groups [x_moe,2],
    queues [8,2], tiles [x_moe*(n1+n2),4]) as numpy arrays."""
    import numpy as np
    lib = load_library()
    counts = np.ascontiguousarray(counts, dtype=np.int32)
    offsets = np.ascontiguousarray(offsets, dtype=np.int32)
    E = len(counts)
    cap = int(sum(-(-int(c) // M_t) for c in counts if c > 0))
    rt = np.zeros((max(cap, 1), 4), np.int32)
    gr = np.zeros((max(cap, 1), 2), np.int32)
    qu = np.zeros((8, 2), np.int32)
    nt = max(cap * (n1 + n2), 1)
    tl = np.zeros((nt, 4), np.int32)
    p = lambda a: a.ctypes.data_as(C.c_void_p)  # noqa: E731
    x = lib.moe_sched_layout(p(counts), p(offsets), E, M_t, gmax, n1, n2, rt.shape[0], p(rt), p(gr), p(qu), nt, p(tl))
    if x < 0:
        raise ValueError(f"moe_sched_layout returned {x}")
    return rt[:x], gr[:x], qu, tl[:x * (n1 + n2)]
