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
    """A copy of the HIP sources under a temporary root that bench.py reads."""
    src = os.path.join(ROOT, "paper_2606_22768_amd", "csrc")
    dst = tmp_path / "paper_2606_22768_amd" / "csrc"
    shutil.copytree(src, dst)
    (tmp_path / "profiles").mkdir()
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    return tmp_path


def _touch(tree, name):
    p = tree / "paper_2606_22768_amd" / "csrc" / name
    p.write_text(p.read_text() + "\n// edited\n")


def test_component_hashes_cover_their_sources(tree):
    step0, js0 = bench.kernel_source_hash("step"), bench.kernel_source_hash("js")
    assert step0 != js0
    _touch(tree, "js.hip")
    step1, js1 = bench.kernel_source_hash("step"), bench.kernel_source_hash("js")
    assert step1 == step0 and js1 != js0           # the JS kernels are not part of the step
    _touch(tree, "engine.hip")
    step2, js2 = bench.kernel_source_hash("step"), bench.kernel_source_hash("js")
    assert step2 != step1 and js2 == js1           # launch code belongs to the step only
    _touch(tree, "kernels.hpp")
    assert bench.kernel_source_hash("step") != step2 and bench.kernel_source_hash("js") != js2


def test_traffic_applies_only_to_the_sources_it_was_taken_on(tree):
    wl, algo = "m8_p1100m_bf16", 123_200_000_000
    assert bench.read_traffic(wl, algo) is None    # no summary
    summary = {"kernel_source_hash": bench.kernel_source_hash("step"), "fetch_bytes_per_launch": 70_400_000_000,
               "write_bytes_per_launch": 52_800_000_000}
    path = tree / "profiles" / f"traffic_fused_step_{wl}.json"
    path.write_text(json.dumps(summary))
    t = bench.read_traffic(wl, algo)
    assert t["total_bytes"] == algo and t["ratio_to_algorithmic"] == pytest.approx(1.0)
    _touch(tree, "js.hip")                         # a JS edit leaves the step's counters valid
    assert bench.read_traffic(wl, algo) is not None
    _touch(tree, "kernels_bf16.hip")               # a step edit voids them
    assert bench.read_traffic(wl, algo) is None
