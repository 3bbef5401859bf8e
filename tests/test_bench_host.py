"""Host-side logic of bench.py (no GPU): the one-GPU contract, which sources
each component's hash covers, and when the committed traffic counters apply."""

import json
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


@pytest.mark.parametrize("argv, env", [(["--gpus", "2"], {}), ([], {"WORLD_SIZE": "2"})])
def test_more_than_one_gpu_is_refused(argv, env):
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *argv], capture_output=True, text=True,
                       env={**os.environ, **env}, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


@pytest.fixture()
def tree(tmp_path, monkeypatch):
    """A copy of the library sources and header under a temporary root that
    bench.py and the build's hash read."""
    shutil.copytree(os.path.join(ROOT, "paper_2606_22768_amd", "csrc"), tmp_path / "paper_2606_22768_amd" / "csrc")
    (tmp_path / "include").mkdir()
    shutil.copy(os.path.join(ROOT, "include", "fgd.h"), tmp_path / "include" / "fgd.h")
    (tmp_path / "profiles").mkdir()
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    return tmp_path


def _touch(tree, name):
    p = tree / "paper_2606_22768_amd" / "csrc" / name
    p.write_text(p.read_text() + "\n// edited\n")


def _hashes(tree):
    from paper_2606_22768_amd import build
    return build.source_hashes(str(tree))


def test_component_hashes_cover_their_sources(tree):
    h0 = _hashes(tree)
    assert h0["step"] != h0["js"]
    _touch(tree, "js.hip")
    h1 = _hashes(tree)
    assert h1["step"] == h0["step"] and h1["js"] != h0["js"] and h1["all"] != h0["all"]  # JS is not the step
    _touch(tree, "js.hpp")
    h1b = _hashes(tree)
    assert h1b["step"] == h1["step"] and h1b["js"] != h1["js"]  # the JS launcher's header
    _touch(tree, "js_api.hip")
    h1c = _hashes(tree)
    assert h1c["step"] == h1b["step"] and h1c["js"] != h1b["js"]  # the JS entry points
    _touch(tree, "api.hpp")
    h1d = _hashes(tree)
    assert h1d["step"] != h1c["step"] and h1d["js"] != h1c["js"]  # the error helpers both use
    h1 = h1d
    _touch(tree, "engine.hip")
    h2 = _hashes(tree)
    assert h2["step"] != h1["step"] and h2["js"] == h1["js"]  # launch code belongs to the step only
    _touch(tree, "kernels.hpp")
    h3 = _hashes(tree)
    assert h3["step"] != h2["step"] and h3["js"] != h2["js"]
    _touch(tree, "topology.cpp")
    h4 = _hashes(tree)
    assert h4["step"] == h3["step"] and h4["all"] != h3["all"]  # host code: only the whole library


def test_traffic_applies_only_to_the_library_it_was_taken_with(tree):
    wl, algo = "m8_p1100m_bf16", 123_200_000_000
    step = _hashes(tree)["step"]
    assert bench.read_traffic(wl, algo, step) is None    # no summary
    summary = {"kernel_source_hash": step, "fetch_bytes_per_launch": 70_400_000_000,
               "write_bytes_per_launch": 52_800_000_000}
    path = tree / "profiles" / f"traffic_fused_step_{wl}.json"
    path.write_text(json.dumps(summary))
    t = bench.read_traffic(wl, algo, step)
    assert t["total_bytes"] == algo and t["ratio_to_algorithmic"] == pytest.approx(1.0)
    _touch(tree, "js.hip")                               # a JS edit leaves the step's counters valid
    assert bench.read_traffic(wl, algo, _hashes(tree)["step"]) is not None
    _touch(tree, "kernels_bf16.hip")                     # a library of edited step sources voids them
    assert bench.read_traffic(wl, algo, _hashes(tree)["step"]) is None
