"""Compile libbpc.so for gfx950 with hipcc (in-tree, next to this file).

    python -m paper_2608_04405_amd.build_lib [--trace]

Each HIP translation unit is compiled in parallel, then linked.  --trace
builds libbpc_trace.so instead: the same library with per-workgroup phase
timestamps (-DBPC_TRACE, bpc_trace_buffer()), for measurement only.  All device
code is built with floating-point contraction off (the code-bit arithmetic
must round after every multiply and add) and with packed-fp32 instructions
disabled.
"""

from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
OUT = os.path.join(HERE, "libbpc.so")
OUT_TRACE = os.path.join(HERE, "libbpc_trace.so")
BUILD_DIR = os.path.join(os.path.dirname(HERE), "_build")
SOURCES = ["bpc_api.hip", "build_kernels.hip", "decode_kernels.hip", "eas_kernels.hip", "hash_mm_kernels.hip"]
ARCH = os.environ.get("BPC_OFFLOAD_ARCH", "gfx950")

COMMON = [
    "-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
    "-ffp-contract=off",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
]


def _hipcc() -> str:
    for cand in (shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def _compile(hipcc: str, src: str, trace: bool) -> str:
    obj = os.path.join(BUILD_DIR, os.path.splitext(src)[0] + ("_trace.o" if trace else ".o"))
    cmd = [hipcc, *COMMON, *(["-DBPC_TRACE"] if trace else []), "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    return obj


def build(verbose: bool = False, trace: bool = False) -> str:
    os.makedirs(BUILD_DIR, exist_ok=True)
    hipcc = _hipcc()
    out = OUT_TRACE if trace else OUT
    with cf.ThreadPoolExecutor(max_workers=len(SOURCES)) as ex:
        objs = list(ex.map(lambda s: _compile(hipcc, s, trace), SOURCES))
    tmp = out + ".tmp"
    cmd = [hipcc, "-shared", "-fPIC", f"--offload-arch={ARCH}", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, out)
    if verbose:
        print(f"built {out}")
    return out


if __name__ == "__main__":
    build(verbose=True, trace="--trace" in sys.argv[1:])
    sys.exit(0)
