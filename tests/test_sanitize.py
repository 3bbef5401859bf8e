"""CPU sanitizer tier: the oracle (oracle/fgd_oracle.c) and the library's
host topology code (paper_2606_22768_amd/csrc/topology.cpp), the two pieces
that parse caller-supplied CSR structures, masks and subset segments, built
with AddressSanitizer and UndefinedBehaviorSanitizer (gcc/g++, host code
only) and run by tests/sanitize/driver.cpp on seeded random and malformed
inputs.  Any out-of-bounds access, leak or undefined operation fails it."""

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = ["-g", "-O1", "-fno-omit-frame-pointer", "-fsanitize=address,undefined", "-fno-sanitize-recover=all"]


@pytest.mark.skipif(shutil.which("g++") is None or shutil.which("gcc") is None, reason="needs gcc and g++")
def test_oracle_and_topology_under_asan_and_ubsan(tmp_path):
    oracle_o, topo_o, exe = tmp_path / "oracle.o", tmp_path / "topology.o", tmp_path / "driver"
    csrc = os.path.join(ROOT, "paper_2606_22768_amd", "csrc")
    cmds = [
        ["gcc", "-std=c11", "-fno-fast-math", "-ffp-contract=off", *SAN, "-c",
         os.path.join(ROOT, "oracle", "fgd_oracle.c"), "-o", str(oracle_o)],
        ["g++", "-std=c++17", *SAN, "-c", os.path.join(csrc, "topology.cpp"), "-o", str(topo_o)],
        ["g++", "-std=c++17", *SAN, "-I", csrc, os.path.join(ROOT, "tests", "sanitize", "driver.cpp"),
         str(oracle_o), str(topo_o), "-o", str(exe), "-lm"],
    ]
    for c in cmds:
        r = subprocess.run(c, capture_output=True, text=True)
        assert r.returncode == 0, (c, r.stderr)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0:halt_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([str(exe)], capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0 and r.stdout.strip().endswith("ok"), (r.returncode, r.stdout[-2000:], r.stderr[-4000:])
