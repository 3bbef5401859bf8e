"""Builds libfgd.so in-tree: hipcc for the gfx950 kernels and the engine,
g++ for the host-only topology code.

    python -m paper_2606_22768_amd.build
"""

from __future__ import annotations

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libfgd.so")

HIP_SOURCES = ["engine.hip", "kernels_f32.hip", "kernels_bf16.hip", "kernels_f32_ms.hip", "kernels_bf16_ms.hip",
               "kernels_f32_split.hip", "kernels_bf16_split.hip", "kernels_common.hip", "js.hip"]
CXX_SOURCES = ["topology.cpp"]

ARCH = "gfx950"
# Packed float32 instructions are kept out of every kernel (the compiler may
# otherwise form v_pk_* from plain float code).
HIP_FLAGS = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}", "-Wall", "-Wno-unused-function",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", "-ffp-contract=fast"]
CXX_FLAGS = ["-O2", "-std=c++17", "-fPIC", "-Wall"]


def _hipcc():
    for c in (shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found")


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"command failed ({r.returncode}): {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    return r


def build(verbose: bool = False, jobs: int = 8, defines=(), out=None, build_dir=None) -> str:
    """Compiles every source and links libfgd.so.  Always recompiles.

    defines: extra -D tuning macros (defaults are the shipped values);
    out / build_dir: where the library and objects go (default in-tree)."""
    lib_path = out or LIB
    bdir = build_dir or BUILD
    os.makedirs(bdir, exist_ok=True)
    extra = [f"-D{d}" for d in defines]
    hipcc = _hipcc()
    inc = ["-I", os.path.join(ROOT, "include")]
    cmds = []
    objs = []
    for s in HIP_SOURCES:
        o = os.path.join(bdir, s.replace(".", "_") + ".o")
        cmds.append([hipcc, *HIP_FLAGS, *extra, *inc, "-c", os.path.join(CSRC, s), "-o", o])
        objs.append(o)
    for s in CXX_SOURCES:
        o = os.path.join(bdir, s.replace(".", "_") + ".o")
        cmds.append(["g++", *CXX_FLAGS, *extra, *inc, "-c", os.path.join(CSRC, s), "-o", o])
        objs.append(o)
    with ThreadPoolExecutor(max_workers=jobs) as ex:
        for r in ex.map(_run, cmds):
            if verbose and r.stderr.strip():
                print(r.stderr, file=sys.stderr)
    tmp = lib_path + ".tmp"
    _run([hipcc, "-shared", "-fPIC", f"--offload-arch={ARCH}", "-o", tmp, *objs])
    os.replace(tmp, lib_path)
    return lib_path


if __name__ == "__main__":
    print(build(verbose=True))
