"""Build libmoe_apk.so (HIP, gfx950) in-tree with hipcc.

    python -m paper_2607_18002_amd.build [--verbose]

Each source compiles to an object under _build/ (in parallel), then hipcc
links the shared library next to this file.  Always rebuilds.
"""
from __future__ import annotations

import argparse
import concurrent.futures as cf
import os
import re
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libmoe_apk.so")
SOURCES = ["api.cpp", "route.hip", "permute.hip", "combine.hip", "ffn.hip", "pack.hip"]
# measurement kernels (achievable MFMA and HBM read peaks), a library of their own
PEAKS_LIB = os.path.join(PKG, "libmoe_peaks.so")
PEAKS_SOURCES = ["peaks.hip"]
# Every source file the persistent FFN kernel is compiled from (hashed to tie
# recorded hardware-counter figures to the kernel they were taken on).
FFN_KERNEL_SOURCES = ["paper_2607_18002_amd/csrc/ffn.hip", "paper_2607_18002_amd/csrc/tile_bf16.hpp",
                      "paper_2607_18002_amd/csrc/tile_bf16_tall.hpp", "paper_2607_18002_amd/csrc/tile_fp8.hpp",
                      "paper_2607_18002_amd/csrc/common.hpp", "paper_2607_18002_amd/csrc/sched_index.hpp",
                      "include/moe_apk.h"]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    # packed fp32 instructions are kept out of the generated code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    f"-I{os.path.join(ROOT, 'include')}", f"-I{CSRC}",
    "-Wall", "-Wno-unused-function", "-Wno-unused-variable",
]


# Per-lane scratch the persistent kernels may use (register spills).  A larger
# figure means the compiler copied the kernel arguments to scratch (an index
# into them that differs per lane, or their address passed to a function it
# did not inline), which slows every tile; the build refuses it.
SCRATCH_LIMIT = {"apk_kernel": 512, "plain_gemm_kernel": 512}


def _scratch_check(src: str, lines) -> None:
    fn = None
    for ln in lines:
        m = re.search(r"Function Name: (\S+)", ln)
        if m:
            fn = m.group(1)
            continue
        m = re.search(r"ScratchSize \[bytes/lane\]: (\d+)", ln)
        if m and fn:
            for key, limit in SCRATCH_LIMIT.items():
                if key in fn and int(m.group(1)) > limit:
                    raise RuntimeError(f"{src}: {fn} uses {m.group(1)} bytes of scratch per lane (limit {limit}): "
                                       "its kernel arguments were copied to scratch")


# data operand: the first of a buffer store, the second of a global, flat or scratch store
_STORE_WIDE = re.compile(r"^(?:buffer_store_dwordx[34]\s+|(?:global|flat|scratch)_store_dwordx[34]\s+\S+,\s*)"
                         r"v\[(\d+):(\d+)\]")
_VREG = re.compile(r"^v\[(\d+):(\d+)\]|^v(\d+)$")


def _vregs(tok: str):
    m = _VREG.match(tok.rstrip(","))
    if not m:
        return set()
    if m.group(3) is not None:
        return {int(m.group(3))}
    return set(range(int(m.group(1)), int(m.group(2)) + 1))


def _store_data_check(src: str, asm: str) -> None:
    """A store of more than 8 bytes reads its data registers after it issues;
    on gfx950 two wait states must pass before a VALU instruction writes them.
    Refuse code in which the next VALU instruction writes them sooner."""
    lines = [ln.strip() for ln in asm.splitlines()]
    for i, t in enumerate(lines):
        m = _STORE_WIDE.match(t)
        if not m:
            continue
        data = set(range(int(m.group(1)), int(m.group(2)) + 1))
        states = 0
        for u in lines[i + 1:i + 12]:
            # labels, comments and directives emit nothing; control falls through a label
            if not u or u.startswith(";") or u.startswith(".") or u.endswith(":"):
                continue
            op = u.split()[0]
            if op in ("s_branch", "s_setpc_b64", "s_endpgm"):
                break
            if op == "s_nop":
                states += int(u.split()[1], 0) + 1
            else:
                if op.startswith("v_") and len(u.split()) > 1 and _vregs(u.split()[1]) & data:
                    raise RuntimeError(f"{src}: '{u}' overwrites the data of '{t}' after {states} wait states (2 needed)")
                states += 1
            if states >= 2:
                break


def _compile_asm_check(src: str, build_dir: str = BUILD, defines=()) -> None:
    asm_path = os.path.join(build_dir, os.path.splitext(src)[0] + ".device.s")
    cmd = [HIPCC, *FLAGS, *[f"-D{d}" for d in defines], "--cuda-device-only", "-S", "-x", "hip",
           os.path.join(CSRC, src), "-o", asm_path]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"device assembly failed: {src}\n" + (r.stdout + r.stderr)[-3000:])
    with open(asm_path) as f:
        _store_data_check(src, f.read())


def _compile(src: str, verbose: bool, build_dir: str = BUILD, defines=()) -> str:
    obj = os.path.join(build_dir, os.path.splitext(src)[0] + ".o")
    cmd = [HIPCC, *FLAGS, *[f"-D{d}" for d in defines], "-x", "hip", "-c", os.path.join(CSRC, src), "-o", obj]
    check = src == "ffn.hip"
    if verbose or check:
        cmd.insert(1, "-Rpass-analysis=kernel-resource-usage")
    r = subprocess.run(cmd, capture_output=True, text=True)
    out = (r.stdout + r.stderr).strip()
    # hipcc's host pass does not know the packed-fp32 feature; that warning is harmless
    lines = [ln for ln in out.splitlines() if "packed-fp32-ops" not in ln and "not a recognized feature" not in ln]
    if r.returncode != 0:
        raise RuntimeError(f"compile failed: {src}\n" + "\n".join(lines))
    if check:
        _scratch_check(src, lines)
    lines = [ln for ln in lines if verbose or "kernel-resource-usage" not in ln]
    if verbose and lines:
        print("\n".join(lines))
    return obj


def ffn_kernel_hash() -> str:
    """sha256 (first 16 hex digits) over the persistent FFN kernel's sources."""
    import hashlib
    h = hashlib.sha256()
    for name in FFN_KERNEL_SOURCES:
        with open(os.path.join(ROOT, name), "rb") as f:
            h.update(name.encode() + b"\0" + f.read())
    return h.hexdigest()[:16]


def _link(objs, lib: str) -> None:
    tmp = lib + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed\n" + r.stdout + r.stderr)
    os.replace(tmp, lib)


def build(verbose: bool = False, out_dir: str = "", defines=()) -> str:
    """Build both libraries in-tree; with out_dir, build only the hot-path
    library there (with extra -D defines), e.g. to compare two builds."""
    if not os.path.exists(HIPCC) and shutil.which("hipcc") is None:
        raise RuntimeError("hipcc not found")
    bdir = os.path.join(out_dir, "_obj") if out_dir else BUILD
    os.makedirs(bdir, exist_ok=True)
    allsrc = SOURCES if out_dir else SOURCES + PEAKS_SOURCES
    with cf.ThreadPoolExecutor(max_workers=8) as ex:
        # every kernel's device code is also checked for the store-data hazard
        asm_checks = [ex.submit(_compile_asm_check, s, bdir, defines) for s in allsrc if s.endswith(".hip")]
        objs = list(ex.map(lambda s: _compile(s, verbose, bdir, defines), allsrc))
        for c in asm_checks:
            c.result()
    lib = os.path.join(out_dir, "libmoe_apk.so") if out_dir else LIB
    _link(objs[:len(SOURCES)], lib)
    if not out_dir:
        _link(objs[len(SOURCES):], PEAKS_LIB)
    return lib


if __name__ == "__main__":
    ap = argparse.ArgumentParser()
    ap.add_argument("--verbose", action="store_true")
    ap.add_argument("--out-dir", default="", help="build only the hot-path library into this directory")
    ap.add_argument("-D", dest="defines", action="append", default=[], help="extra preprocessor define")
    args = ap.parse_args()
    path = build(args.verbose, args.out_dir, args.defines)
    print(path)
    sys.exit(0)
