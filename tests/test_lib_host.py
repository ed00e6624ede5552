"""CPU-only checks of the C-ABI library: it loads, exports every symbol the
header declares, its struct layouts match the binding, its host helpers agree
with the oracle's Eq. (3)/(4), and argument errors are reported before any
device work."""
import ctypes as C
import os
import re

import numpy as np
import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "moe_apk.h")
LIB = os.path.join(ROOT, "paper_2607_18002_amd", "libmoe_apk.so")

pytestmark = pytest.mark.skipif(not os.path.exists(LIB), reason="library not built (run __graft_entry__.build())")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = re.findall(r"^\s*[A-Za-z_][\w\s\*]*?\b(moe_\w+)\s*\(", text, flags=re.M)
    return sorted(set(names))


def test_header_declares_the_four_calls():
    names = declared_functions()
    for n in ("moe_topk_route", "moe_permute", "moe_grouped_ffn_persistent", "moe_combine"):
        assert n in names


def test_exports_every_declared_symbol():
    lib = C.CDLL(LIB)
    missing = [n for n in declared_functions() if not hasattr(lib, n)]
    assert not missing, missing


def test_binding_layouts_match_library():
    from paper_2607_18002_amd import _lib
    lib = _lib.load_library()
    assert lib.moe_abi_sizeof(0) == C.sizeof(_lib.OpDesc)
    assert lib.moe_abi_sizeof(1) == C.sizeof(_lib.SchedConfig)
    assert lib.moe_abi_sizeof(2) == C.sizeof(_lib.TraceRec) == 80
    assert lib.moe_abi_sizeof(3) == C.sizeof(_lib.OpStats) == 48
    assert lib.moe_abi_sizeof(4) == C.sizeof(_lib.RouteArgs)
    assert lib.moe_abi_sizeof(5) == C.sizeof(_lib.PermuteArgs)
    assert lib.moe_abi_sizeof(6) == C.sizeof(_lib.CombineArgs)
    assert lib.moe_abi_sizeof(9) == 0


def test_status_strings():
    from paper_2607_18002_amd import ops
    assert ops.status_string(0) == "MOE_OK"
    assert ops.status_string(-3) == "MOE_ERR_CAPACITY"
    assert ops.status_string(-7) == "MOE_ERR_BAD_EXPERT"
    assert ops.status_string(-8) == "MOE_ERR_INTERNAL"


def test_x_moe_matches_oracle():
    from paper_2607_18002_amd import ops
    rng = np.random.default_rng(3)
    for _ in range(50):
        counts = rng.integers(0, 700, size=int(rng.integers(1, 40)))
        counts[rng.random(len(counts)) < 0.2] = 0
        mt = int(rng.choice([1, 16, 32, 128, 256]))
        assert ops.moe_x_moe(counts, mt) == oracle.x_moe(counts, mt)


def test_decode_quota_matches_oracle():
    from paper_2607_18002_amd import ops
    rng = np.random.default_rng(4)
    for _ in range(500):
        q = int(rng.integers(0, 257))
        x = int(rng.integers(0, 400))
        xs = int(rng.integers(-2, 300))
        qmax = int(rng.integers(1, 257))
        c = int(rng.choice([1, 2, 8, 16]))
        assert ops.moe_decode_quota(q, x, xs, qmax, c) == oracle.decode_quota(q, x, xs, qmax, c)


def test_row_align_and_workspace_queries():
    from paper_2607_18002_amd import _lib, ops
    # segments are aligned to one 32-row MFMA block; tiles are at most bm rows
    for ph in (_lib.MOE_PREFILL, _lib.MOE_DECODE):
        for dt in (_lib.MOE_BF16, _lib.MOE_FP8_E4M3):
            assert ops.moe_ffn_row_align(ph, dt) == 32
    assert ops.moe_ffn_tile_shape(_lib.MOE_PREFILL, _lib.MOE_BF16) == (192, 256, 64)   # tall prefill tile
    assert ops.moe_ffn_tile_shape(_lib.MOE_DECODE, _lib.MOE_BF16) == (128, 256, 64)
    assert ops.moe_ffn_tile_shape(_lib.MOE_PREFILL, _lib.MOE_FP8_E4M3) == (128, 256, 128)
    assert ops.moe_ffn_row_align(7, _lib.MOE_BF16) < 0
    for ph in (_lib.MOE_PREFILL, _lib.MOE_DECODE):
        bm, bn, bk = ops.moe_ffn_tile_shape(ph, _lib.MOE_BF16)
        assert bm % ops.moe_ffn_row_align(ph, _lib.MOE_BF16) == 0 and bn % 64 == 0 and bk % 16 == 0
    assert ops.moe_permute_workspace_bytes(16384, 8, 32) >= 32 * 32 * 4
    d = _lib.OpDesc(capacity=69600, row_align=32)
    cfg = _lib.SchedConfig()
    assert ops.moe_ffn_workspace_bytes([d], cfg) >= 2 * (69600 // 128) * 4


def test_argument_errors_before_any_launch():
    """Invalid arguments are rejected on the host with a message and never
    reach the device (this container has no GPU)."""
    from paper_2607_18002_amd import _lib
    lib = _lib.load_library()
    assert lib.moe_topk_route(None, -1, 8, 2, 0, 8, None, None, None) == _lib.MOE_ERR_INVALID_ARG
    assert b"T=-1" in lib.moe_last_error()
    assert lib.moe_topk_route(None, 4, 2000, 2, 0, 8, None, None, None) == _lib.MOE_ERR_UNSUPPORTED
    assert lib.moe_topk_route(None, 4, 8, 9, 0, 8, None, None, None) == _lib.MOE_ERR_INVALID_ARG
    assert lib.moe_topk_route(None, 0, 8, 2, 0, 8, None, None, None) == _lib.MOE_OK     # T == 0: nothing to do
    args = [None, 10, 8, 4, None, _lib.MOE_BF16, None, 256, 128, 10] + [None] * 9
    assert lib.moe_permute(*args) == _lib.MOE_ERR_CAPACITY          # capacity 10 < 10*4 + 4*127
    args[7] = 100                                                    # H not a multiple of 128
    assert lib.moe_permute(*args) == _lib.MOE_ERR_UNSUPPORTED
    assert lib.moe_combine(None, None, None, 4, 2, 12, None, _lib.MOE_BF16, None) == _lib.MOE_ERR_UNSUPPORTED
    assert lib.moe_combine(None, None, None, 4, 2, 16, None, 7, None) == _lib.MOE_ERR_UNSUPPORTED
    assert lib.moe_grouped_ffn_persistent(None, 1, None, None, None, None) == _lib.MOE_ERR_INVALID_ARG


def test_masked_route_argument_errors():
    """The masked-layout fields of moe_topk_route_batch are checked on the host
    before anything is launched: 1 <= T, slots a multiple of 32 and >= T,
    both maps and the placement workspace given and aligned, E_local within
    the placement's limit."""
    from paper_2607_18002_amd import _lib
    lib = _lib.load_library()
    fake = 0x10000                                          # never dereferenced: the call fails first

    def call(**kw):
        a = dict(logits=fake, T=64, E_global=64, top_k=4, local_begin=0, E_local=8, topk_ids=fake, topk_w=fake,
                 slots=64, counts=fake, place_ws=fake + 256, assign_to_row=fake, row_to_assign=fake)
        a.update(kw)
        arr = (_lib.RouteArgs * 1)(_lib.RouteArgs(**a))
        return lib.moe_topk_route_batch(arr, 1, None)

    assert call(slots=40) == _lib.MOE_ERR_INVALID_ARG            # not a multiple of 32
    assert b"slots (40)" in lib.moe_last_error()
    assert call(slots=32) == _lib.MOE_ERR_INVALID_ARG            # fewer slots than tokens
    assert call(assign_to_row=None) == _lib.MOE_ERR_INVALID_ARG
    assert call(place_ws=None) == _lib.MOE_ERR_INVALID_ARG
    assert call(place_ws=fake + 4) == _lib.MOE_ERR_INVALID_ARG   # not 8-byte aligned
    assert call(T=0, slots=0) == _lib.MOE_ERR_INVALID_ARG         # a masked entry needs a token
    assert call(E_local=1025, E_global=2048) != _lib.MOE_OK
    assert call(counts=None, place_ws=None) != _lib.MOE_ERR_INVALID_ARG   # unmasked entry passes the checks


def test_route_place_workspace_bytes():
    """One 64-bit record per (chunk, local expert) after a 256-byte header;
    chunks of 4 tokens up to 2048 tokens, of 16 above."""
    from paper_2607_18002_amd import ops
    assert ops.moe_route_place_workspace_bytes(0, 32) == 0
    assert ops.moe_route_place_workspace_bytes(1, 32) == 256 + 32 * 8
    assert ops.moe_route_place_workspace_bytes(1024, 32) == 256 + 256 * 32 * 8
    assert ops.moe_route_place_workspace_bytes(1025, 8) == 256 + 257 * 8 * 8
    assert ops.moe_route_place_workspace_bytes(2049, 8) == 256 + 512 * 8 * 8     # covers T = 2048 in 4-token chunks
    assert ops.moe_route_place_workspace_bytes(16384, 8) == 256 + 1024 * 8 * 8


def test_split_trace_blocks():
    """Trace buffers hold one block per workgroup; a block ends at its first
    op = -1 record or at its end, and the records come back in start order."""
    from paper_2607_18002_amd.pipeline import TRACE_DTYPE, split_trace
    recs = np.zeros(12, dtype=TRACE_DTYPE)
    recs["op"] = -7                                           # stale contents past a terminator
    # block 0 (records 0-3): two tiles then the terminator
    recs["op"][0:2] = 0
    recs["t_start"][0:2] = [30, 10]
    recs["op"][2] = -1
    # block 1 (records 4-7): full, no terminator
    recs["op"][4:8] = 1
    recs["t_start"][4:8] = [5, 15, 25, 35]
    # block 2 (records 8-11): terminator first
    recs["op"][8] = -1
    got = split_trace(recs, 3)
    assert got["t_start"].tolist() == [5, 10, 15, 25, 30, 35]
    assert got["op"].tolist() == [1, 0, 1, 1, 0, 1]
    assert len(split_trace(recs[:0], 3)) == 0
