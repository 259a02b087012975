"""Build libframeft.so for gfx950 with hipcc (in-tree, next to this file).

Usage: python -m paper_2608_26430_amd.build  (or build() from Python).
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
BUILD_DIR = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libframeft.so")
# (source, object name, extra flags): the generic kernels are instantiated by one source compiled
# once per direction and activation type, so that their long compiles run in parallel
SOURCES = [("capi.cpp", "capi.cpp.o", []), ("framegen.cpp", "framegen.cpp.o", []), ("plan.cpp", "plan.cpp.o", []),
           ("kernels.hip", "kernels.hip.o", []), ("kernels_w128.hip", "kernels_w128.hip.o", []),
           ("optim.hip", "optim.hip.o", []), ("group.cpp", "group.cpp.o", []),
           ("lift.hip", "lift.hip.o", [])] + [
    ("gen_inst.hip", f"gen_{d}_{t}{'_ms' if ms else ''}.o",
     [f"-DGEN_BWD={int(d == 'bwd')}", f"-DGEN_BF16={int(t == 'bf16')}", f"-DGEN_MS={ms}"])
    for d in ("bwd", "fwd") for t in ("bf16", "f32") for ms in (0, 1)]

ARCH = "gfx950"
COMMON = [
    "-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}", "-fno-strict-aliasing",
    # Packed fp32 VALU forms are kept out of the generated code.
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-result", "-Wno-unused-function",
    "-I", os.path.join(ROOT, "include"),
]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def _compile(entry) -> str:
    src, name, flags = entry
    obj = os.path.join(BUILD_DIR, name)
    cmd = [hipcc(), *COMMON, *flags, "-c", os.path.join(CSRC, src), "-o", obj]
    if src.endswith(".cpp"):
        cmd[1:1] = ["-x", "hip"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    noise = "'-packed-fp32-ops' is not a recognized feature"
    msgs = "\n".join(l for l in (r.stdout + r.stderr).splitlines() if noise not in l)
    if r.returncode != 0:
        raise RuntimeError(f"compiling {src} failed:\n{' '.join(cmd)}\n{msgs}")
    if msgs.strip():
        print(msgs, file=sys.stderr)
    return obj


def build(verbose: bool = True) -> str:
    """Compile every source and link libframeft.so; always rebuilds."""
    os.makedirs(BUILD_DIR, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=min(max(2, (os.cpu_count() or 4) - 1), len(SOURCES))) as ex:
        objs = list(ex.map(_compile, SOURCES))
    tmp = LIB + ".tmp"
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-Wl,--no-undefined", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"linking failed:\n{' '.join(cmd)}\n{r.stdout}{r.stderr}")
    os.replace(tmp, LIB)
    if verbose:
        print(f"built {LIB}")
    return LIB


if __name__ == "__main__":
    build()
