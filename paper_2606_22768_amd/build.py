"""Builds libfgd.so in-tree: hipcc for the gfx950 kernels and the engine,
g++ for the host-only topology code.

    python paper_2606_22768_amd/build.py

(run as a script: importing the package loads the library, which a stale
or missing build would refuse).

The library carries the hashes of the sources it was built from: they are
compiled into it (fgd_source_hash) and written beside it in libfgd.so.json,
so a library and a source tree that disagree can be told apart without
running anything (needs_build) and once loaded (the binding refuses such a
library).
"""

from __future__ import annotations

import hashlib
import json
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
               "kernels_f32_split.hip", "kernels_bf16_split.hip", "kernels_wg.hip", "kernels_common.hip",
               "js.hip", "js_api.hip"]
CXX_SOURCES = ["topology.cpp"]

ARCH = "gfx950"
# Packed float32 instructions are kept out of every kernel (the compiler may
# otherwise form v_pk_* from plain float code).
HIP_FLAGS = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}", "-Wall", "-Wno-unused-function",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", "-ffp-contract=fast"]
CXX_FLAGS = ["-O2", "-std=c++17", "-fPIC", "-Wall"]

HASH_COMPONENTS = ("all", "step", "js")


def source_hashes(root: str = ROOT) -> dict:
    """Hashes (16 hex digits) of the sources under `root`:
    all   every file under paper_2606_22768_amd/csrc and include/fgd.h;
    step  the HIP sources of the outer step, its split halves, consensus,
          finalize and copy kernels and their launches (every .hip/.hpp but
          the JS distance's js.hip, js.hpp and js_api.hip);
    js    the JS distance kernels, their launcher header, their C entry
          points and the headers those include (kernels.hpp, api.hpp).
    Traffic counters and timings are valid only for the hash they were
    taken with."""
    csrc = os.path.join(root, "paper_2606_22768_amd", "csrc")
    names = sorted(os.listdir(csrc))
    hs = {c: hashlib.sha256() for c in HASH_COMPONENTS}
    for name in names:
        with open(os.path.join(csrc, name), "rb") as f:
            data = name.encode() + b"\0" + f.read()
        hs["all"].update(data)
        if name.endswith((".hip", ".hpp")):
            if name not in ("js.hip", "js.hpp", "js_api.hip"):
                hs["step"].update(data)
            if name in ("js.hip", "js.hpp", "js_api.hip", "kernels.hpp", "api.hpp"):
                hs["js"].update(data)
    with open(os.path.join(root, "include", "fgd.h"), "rb") as f:
        hs["all"].update(b"fgd.h\0" + f.read())
    return {c: h.hexdigest()[:16] for c, h in hs.items()}


def sidecar_path(lib_path: str = LIB) -> str:
    return lib_path + ".json"


def read_sidecar(lib_path: str = LIB):
    """The source hashes recorded beside a built library, or None."""
    try:
        with open(sidecar_path(lib_path)) as f:
            return json.load(f).get("source_hash")
    except (OSError, ValueError):
        return None


def needs_build(lib_path: str = LIB, root: str = ROOT) -> bool:
    """True when the library is missing or was built from other sources than
    those now under `root` (judged from its sidecar, without loading it)."""
    if not os.path.exists(lib_path):
        return True
    return read_sidecar(lib_path) != source_hashes(root)


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
    hashes = source_hashes()
    extra = [f"-D{d}" for d in defines]
    stamp = [f'-DFGD_HASH_{c.upper()}="{hashes[c]}"' for c in HASH_COMPONENTS]
    hipcc = _hipcc()
    inc = ["-I", os.path.join(ROOT, "include")]
    cmds = []
    objs = []
    for s in HIP_SOURCES:
        o = os.path.join(bdir, s.replace(".", "_") + ".o")
        cmds.append([hipcc, *HIP_FLAGS, *extra, *(stamp if s == "engine.hip" else []), *inc, "-c",
                     os.path.join(CSRC, s), "-o", o])
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
    # The sidecar is written only with the library it describes: a build
    # with tuning macros is not the shipped configuration, so its sidecar
    # records them and never matches needs_build's plain source hashes.
    side = {"source_hash": hashes if not defines else {**hashes, "defines": list(defines)}}
    with open(sidecar_path(lib_path) + ".tmp", "w") as f:
        json.dump(side, f)
    os.replace(tmp, lib_path)
    os.replace(sidecar_path(lib_path) + ".tmp", sidecar_path(lib_path))
    return lib_path


if __name__ == "__main__":
    print(build(verbose=True))
