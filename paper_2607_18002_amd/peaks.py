"""Achievable peaks of the GPU this runs on, measured with the kernels of
libmoe_peaks.so (csrc/peaks.hip): the bf16 and fp8 MFMA throughput of a loop
of nothing but independent MFMAs on every SIMD, and the HBM read rate of a
streaming read of a buffer far larger than the caches, and the vendor
library's dense bf16 GEMM at an expert GEMM's shape.  Used as context beside
the vendor peaks (bench.py reports the hot path's kernel against both).

    python -m paper_2607_18002_amd.peaks
"""
from __future__ import annotations

import ctypes as C
import json
import os

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libmoe_peaks.so")
_LIB = None

FLOP_PER_MFMA = {1: 32 * 32 * 16 * 2, 2: 32 * 32 * 64 * 2}
CHAINS = 8


def _lib():
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build with `python -m paper_2607_18002_amd.build`")
        lib = C.CDLL(LIB_PATH)
        lib.moe_peak_mfma.restype = C.c_int32
        lib.moe_peak_mfma.argtypes = [C.c_int32, C.c_int32, C.c_int32, C.c_void_p, C.c_void_p]
        lib.moe_peak_stream_read.restype = C.c_int32
        lib.moe_peak_stream_read.argtypes = [C.c_void_p, C.c_int64, C.c_int32, C.c_void_p, C.c_void_p]
        _LIB = lib
    return _LIB


def _time(fn, reps: int):
    import torch
    s = torch.cuda.current_stream()
    fn()                                                      # warm-up (and clock ramp)
    fn()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    ev[0].record(s)
    for _ in range(reps):
        fn()
    ev[1].record(s)
    torch.cuda.synchronize()
    return ev[0].elapsed_time(ev[1]) / reps * 1e-3          # seconds per call


def mfma_tflops(dtype: int = 1, blocks: int = 1024, iters: int = 4000, reps: int = 5) -> float:
    import torch
    out = torch.empty(blocks * 256, dtype=torch.float32, device="cuda")
    s = int(torch.cuda.current_stream().cuda_stream)

    def run():
        if _lib().moe_peak_mfma(dtype, blocks, iters, out.data_ptr(), s) != 0:
            raise RuntimeError("moe_peak_mfma failed")
    t = _time(run, reps)
    return blocks * 4 * iters * CHAINS * FLOP_PER_MFMA[dtype] / t / 1e12


def stream_read_gbs(gib: float = 4.0, blocks: int = 2048, reps: int = 5) -> float:
    import torch
    n = int(gib * (1 << 30)) // 16 * 16
    buf = torch.empty(n, dtype=torch.uint8, device="cuda")
    buf.fill_(1)
    sink = torch.empty(blocks, dtype=torch.int32, device="cuda")
    s = int(torch.cuda.current_stream().cuda_stream)

    def run():
        if _lib().moe_peak_stream_read(buf.data_ptr(), n, blocks, sink.data_ptr(), s) != 0:
            raise RuntimeError("moe_peak_stream_read failed")
    t = _time(run, reps)
    del buf
    return n / t / 1e9


def vendor_gemm_tflops(M: int = 16384, N: int = 3072, K: int = 3072, reps: int = 20) -> float:
    """bf16 dense GEMM throughput of the vendor library (torch.matmul on
    contiguous operands, hipBLASLt) at one expert GEMM's shape with all routed
    rows in one matrix: what a library GEMM reaches without grouping, gating or
    scheduling, as context for the grouped kernel's MFMA fraction."""
    import torch
    g = torch.Generator(device="cuda").manual_seed(0)
    a = torch.randn((M, K), generator=g, device="cuda").to(torch.bfloat16)
    b = torch.randn((K, N), generator=g, device="cuda").to(torch.bfloat16)
    t = _time(lambda: torch.matmul(a, b), reps)
    del a, b
    return 2.0 * M * N * K / t / 1e12


def measure() -> dict:
    return {"mfma_bf16_tflops": round(mfma_tflops(1), 1), "mfma_fp8_tflops": round(mfma_tflops(2), 1),
            "hbm_read_gbs": round(stream_read_gbs(), 1),
            "vendor_gemm_bf16_16384x3072x3072_tflops": round(vendor_gemm_tflops(), 1)}


if __name__ == "__main__":
    print(json.dumps(measure()))
