"""Build libsparseinfer.so (HIP, gfx950) in-tree with hipcc.

Usage: ``python -m paper_2411_12692_amd.build`` (or ``__graft_entry__.build()``).
``python -m paper_2411_12692_amd.build --trace`` builds the phase-trace
variant ``libsparseinfer_trace.so`` instead (the row-owning kernel compiled
with ``-DSI_TRACE``, read by ``paper_2411_12692_amd.phase_trace``).
"""

from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libsparseinfer.so")
TRACE_LIB = os.path.join(PKG, "libsparseinfer_trace.so")
TRACED = "owned.hip"  # the source compiled with -DSI_TRACE in the trace variant
SOURCES = ["api.hip", "pack.hip", "predict.hip", "mlp.hip", "layer.hip", "owned.hip", "diag.hip"]
ARCH = "gfx950"

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc" if os.path.exists("/opt/rocm/bin/hipcc") else "hipcc")

# Packed-FP32 instructions are disabled: compile plain scalar float code only.
COMMON = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-munsafe-fp-atomics",
    "-I", os.path.join(ROOT, "include"),
]


def _run(cmd):
    p = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(l for l in p.stdout.splitlines() if "packed-fp32-ops" not in l)
    if p.returncode != 0:
        raise RuntimeError(f"command failed ({p.returncode}): {' '.join(cmd)}\n{out}")
    return out


def build(verbose: bool = False, trace: bool = False) -> str:
    """Compile every HIP source and link the shared library (``trace``: the
    phase-trace variant); returns its path."""
    out_dir = os.path.join(BUILD, "trace") if trace else BUILD
    lib = TRACE_LIB if trace else LIB
    os.makedirs(out_dir, exist_ok=True)
    objs = []
    jobs = []
    with cf.ThreadPoolExecutor(max_workers=min(8, len(SOURCES))) as ex:
        for src in SOURCES:
            obj = os.path.join(out_dir, os.path.splitext(src)[0] + ".o")
            objs.append(obj)
            extra = ["-DSI_TRACE"] if trace and src == TRACED else []
            cmd = [HIPCC, *COMMON, *extra, "-c", os.path.join(CSRC, src), "-o", obj]
            jobs.append(ex.submit(_run, cmd))
        for j in jobs:
            out = j.result()
            if verbose and out.strip():
                print(out)
    tmp = lib + ".tmp"
    _run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp])
    shutil.move(tmp, lib)
    return lib


if __name__ == "__main__":
    path = build(verbose=True, trace="--trace" in sys.argv[1:])
    print(path)
    sys.exit(0)
