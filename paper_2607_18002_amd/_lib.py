"""ctypes view of libmoe_apk.so: struct layouts and function prototypes that
mirror include/moe_apk.h.  Loading fails loudly when the library is missing;
there is no fallback implementation."""
from __future__ import annotations

import ctypes as C
import os

PKG = os.path.dirname(os.path.abspath(__file__))
# MOE_APK_LIBRARY: path of another build of the library to load instead (to
# compare builds in one process environment); default: the in-tree build.
LIB_PATH = os.environ.get("MOE_APK_LIBRARY") or os.path.join(PKG, "libmoe_apk.so")

MOE_OK = 0
MOE_ERR_INVALID_ARG = -1
MOE_ERR_UNSUPPORTED = -2
MOE_ERR_CAPACITY = -3
MOE_ERR_HIP = -4
MOE_ERR_ABORTED = -5
MOE_ERR_TIMEOUT = -6
MOE_ERR_BAD_EXPERT = -7
MOE_ERR_INTERNAL = -8

MOE_F32, MOE_BF16, MOE_FP8_E4M3 = 0, 1, 2
MOE_PREFILL, MOE_DECODE = 0, 1
MOE_LAYOUT_ROWMAJOR, MOE_LAYOUT_PACKED = 0, 1
MOE_MAX_OPS = 16

_p = C.c_void_p
_i32 = C.c_int32
_i64 = C.c_int64


class OpDesc(C.Structure):
    _fields_ = [
        ("phase", _i32), ("layer", _i32), ("E_local", _i32), ("H", _i32), ("I", _i32),
        ("capacity", _i32), ("row_align", _i32), ("dtype", _i32),
        ("counts", _p), ("offsets", _p), ("x_perm", _p), ("x_perm_scales", _p),
        ("w_gate_up", _p), ("w_gate_up_scales", _p), ("w_down", _p), ("w_down_scales", _p),
        ("h", _p), ("h_scales", _p), ("y_perm", _p),
        ("release_word", _p), ("release_after_ns", _i64),
        ("depends_on_op", _i32), ("weight_layout", _i32), ("gap_ns", _i64),
        ("done_word", _p),
        ("x", _p), ("x_scales", _p), ("row_to_assign", _p), ("T", _i32), ("top_k", _i32),
        ("assign_to_row", _p), ("topk_w", _p), ("y", _p), ("y_dtype", _i32), ("reserved_c", _i32),
    ]


class SchedConfig(C.Structure):
    _fields_ = [
        ("n_workgroups", _i32), ("decode_quota_wg", _i32), ("decode_quota_max_wg", _i32),
        ("x_moe_expected", _i32), ("round_multiple", _i32), ("group_row_tiles", _i32),
        ("abort_word", _p), ("trace", _p), ("trace_capacity", _i64), ("op_stats", _p),
        ("spin_limit", _i64), ("static_partition", _i32), ("prefill_tile_rows", _i32),
    ]


class TraceRec(C.Structure):
    _fields_ = [
        ("op", C.c_int16), ("stage", C.c_int16), ("wg", C.c_int16), ("xcc", C.c_int16),
        ("expert", _i32), ("mblk", _i32), ("nblk", C.c_int16), ("rows", C.c_int16),
        ("quota_seen", C.c_int16), ("phases_seen", C.c_uint8), ("how", C.c_uint8),
        ("t_boundary", C.c_uint64), ("t_polled", C.c_uint64), ("t_claim", C.c_uint64),
        ("t_start", C.c_uint64), ("t_end", C.c_uint64), ("c_start", C.c_uint64), ("c_end", C.c_uint64),
    ]


class OpStats(C.Structure):
    _fields_ = [
        ("t_seen", C.c_uint64), ("t_ready", C.c_uint64), ("t_first", C.c_uint64), ("t_done", C.c_uint64),
        ("x_moe", _i32), ("n_tiles", _i32), ("quota", _i32), ("reserved", _i32),
    ]


class RouteArgs(C.Structure):
    _fields_ = [
        ("logits", _p), ("T", _i32), ("E_global", _i32), ("top_k", _i32), ("local_begin", _i32),
        ("E_local", _i32), ("topk_ids", _p), ("topk_w", _p),
        ("slots", _i32), ("pad0", _i32), ("counts", _p), ("place_ws", _p), ("assign_to_row", _p), ("row_to_assign", _p),
        ("error_flag", _p),
    ]


class PermuteArgs(C.Structure):
    _fields_ = [
        ("topk_ids", _p), ("T", _i32), ("top_k", _i32), ("E_local", _i32), ("x_dtype", _i32),
        ("x", _p), ("x_scales", _p), ("H", _i32), ("row_align", _i32), ("capacity", _i32), ("pad0", _i32),
        ("counts", _p), ("offsets", _p), ("row_to_assign", _p), ("assign_to_row", _p), ("x_perm", _p),
        ("x_perm_scales", _p), ("workspace", _p), ("error_flag", _p),
    ]


class CombineArgs(C.Structure):
    _fields_ = [
        ("y_perm", _p), ("assign_to_row", _p), ("topk_w", _p), ("T", _i32), ("top_k", _i32), ("H", _i32),
        ("y_dtype", _i32), ("y", _p),
    ]


# name -> (restype, argtypes)
PROTOTYPES = {
    "moe_topk_route": (_i32, [_p, _i32, _i32, _i32, _i32, _i32, _p, _p, _p]),
    "moe_topk_route_batch": (_i32, [C.POINTER(RouteArgs), _i32, _p]),
    "moe_permute_batch": (_i32, [C.POINTER(PermuteArgs), _i32, _p]),
    "moe_combine_batch": (_i32, [C.POINTER(CombineArgs), _i32, _p]),
    "moe_permute_workspace_bytes": (C.c_size_t, [_i32, _i32, _i32]),
    "moe_route_place_workspace_bytes": (C.c_size_t, [_i32, _i32]),
    "moe_permute": (_i32, [_p, _i32, _i32, _i32, _p, _i32, _p, _i32, _i32, _i32,
                           _p, _p, _p, _p, _p, _p, _p, _p, _p]),
    "moe_ffn_row_align": (_i32, [_i32, _i32]),
    "moe_ffn_tile_shape": (_i32, [_i32, _i32, C.POINTER(_i32), C.POINTER(_i32), C.POINTER(_i32)]),
    "moe_ffn_workspace_bytes": (C.c_size_t, [C.POINTER(OpDesc), _i32, C.POINTER(SchedConfig)]),
    "moe_grouped_ffn_persistent": (_i32, [C.POINTER(OpDesc), _i32, C.POINTER(SchedConfig), _p, _p, _p]),
    "moe_grouped_ffn_persistent_noalloc": (_i32, [C.POINTER(OpDesc), _i32, C.POINTER(SchedConfig), _p, _p]),
    "moe_grouped_ffn_plain": (_i32, [C.POINTER(OpDesc), _i32, _p, _p, _p]),
    "moe_combine": (_i32, [_p, _p, _p, _i32, _i32, _i32, _p, _i32, _p]),
    "moe_pack_weights": (_i32, [_p, _p, _i32, _i32, _i32, _i32, _p]),
    "moe_x_moe": (_i32, [C.POINTER(_i32), _i32, _i32]),
    "moe_decode_quota": (_i32, [_i32, _i32, _i32, _i32, _i32]),
    "moe_sched_layout": (_i32, [_p, _p, _i32, _i32, _i32, _i32, _i32, _i32, _p, _p, _p, _i64, _p]),
    "moe_abi_sizeof": (C.c_size_t, [_i32]),
    "moe_status_string": (C.c_char_p, [_i32]),
    "moe_last_error": (C.c_char_p, []),
}

_LIB = None


def load_library(path: str = LIB_PATH) -> C.CDLL:
    """Load the HIP library (once).  Raises if it has not been built."""
    global _LIB
    if _LIB is not None:
        return _LIB
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with `python -m paper_2607_18002_amd.build` "
                           "(there is no fallback implementation)")
    lib = C.CDLL(path)
    for name, (res, args) in PROTOTYPES.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    for which, cls in enumerate((OpDesc, SchedConfig, TraceRec, OpStats, RouteArgs, PermuteArgs, CombineArgs)):
        if lib.moe_abi_sizeof(which) != C.sizeof(cls):
            raise RuntimeError(f"ABI mismatch: sizeof({cls.__name__}) is {C.sizeof(cls)} in Python, "
                               f"{lib.moe_abi_sizeof(which)} in the library")
    _LIB = lib
    return lib


class MoEError(RuntimeError):
    def __init__(self, status: int, where: str, msg: str = ""):
        self.status = status
        lib = load_library()
        name = lib.moe_status_string(status).decode()
        super().__init__(f"{where}: {name} ({status}) {msg}".rstrip())


def check(status: int, where: str) -> None:
    if status != MOE_OK:
        lib = load_library()
        raise MoEError(status, where, lib.moe_last_error().decode())
