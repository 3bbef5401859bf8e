"""bench.py end to end on a small workload: one JSON line with the fields the
benchmark contract names, a roofline object priced against HBM, and the
oracle's CPU baseline beside it."""

import json
import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _bench(*argv):
    print(f"[bench-contract] bench.py {' '.join(argv)}", flush=True)
    r = subprocess.run([sys.executable, "-u", os.path.join(ROOT, "bench.py"), *argv], capture_output=True, text=True,
                       timeout=240)
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [ln for ln in r.stdout.splitlines() if ln.strip()]
    assert len(lines) == 1, r.stdout
    return json.loads(lines[0])


def test_fused_bench_line():
    d = _bench("--workload", "tiny_m4_p1m_f32", "--steps", "25", "--warmup", "2", "--copy-gb", "0.05",
               "--cpu-slice", "65536")
    for key in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "higher_is_better", "scaling",
                "vs_baseline", "dtype", "data", "config", "roofline", "cpu_baseline"):
        assert key in d, key
    assert d["n_gpus"] == 1 and d["steps"] == 25 and d["warmup"] == 2
    assert d["unit"] == "GB/s" and d["higher_is_better"] is True and d["data"] == "synthetic"
    assert d["value"] > 0 and d["ms_per_step"] > 0
    assert d["config"]["workload"] == "tiny_m4_p1m_f32"
    assert d["config"]["placement"].startswith("momentum one physical-memory range")  # the default, spread
    # 4 workers x 2^20 float32 parameters: 3 reads + 2 writes of 4 bytes per element-worker
    assert d["config"]["algorithmic_bytes_per_step"] == 4 * (1 << 20) * 20
    r = d["roofline"]
    assert r["bound"] == "hbm" and r["unit"] == "GB/s" and r["peak"] == 8000.0
    assert r["timed_launches"] == 25                   # every timed step, across the restore chunks
    assert r["frac"] == pytest.approx(r["achieved"] / r["peak"], rel=1e-3)
    assert r["bytes_per_launch"] == d["config"]["algorithmic_bytes_per_step"]
    # HBM bytes per launch from committed counters of these sources, or null
    assert r["traffic"] is None or (isinstance(r["traffic"], int) and r["traffic"] == r["traffic_detail"]["total_bytes"])
    c = d["cpu_baseline"]
    assert c["kind"] == "oracle" and c["cores"] == 1 and c["value"] > 0 and c["unit"] == "GB/s"
    pr = d["pattern_reference"]                       # the step's access pattern without arithmetic
    assert pr["ms"] > 0 and pr["gbs"] > 0 and pr["kernel_rate_vs_pattern"] > 0


def test_js_bench_line_is_one_json_object():
    pytest.importorskip("torch")
    d = _bench("--mode", "js", "--steps", "2", "--warmup", "1", "--no-cpu-baseline")
    assert d["mode"] == "js" and d["unit"] == "GB/s" and d["value"] > 0
    assert d["config"]["vocab"] == 128256 and d["config"]["top_k"] == 100
    assert 0.0 < d["cd_js"] < 1.0
    r = d["roofline"]
    assert r["bound"] == "hbm" and r["unit"] == "GB/s" and r["peak"] == 8000.0
    assert r["bytes_per_launch"] == 9 * 2048 * 128256 * 2 and 0.0 < r["frac"] <= 1.0
    assert abs(r["achieved"] - r["bytes_per_launch"] / (r["kernel_avg_ms"] * 1e6)) <= 1e-3 * r["achieved"] + 0.01
    pr = d["pattern_reference"]                       # the row kernel's loads without arithmetic
    assert pr["ms"] > 0 and pr["gbs"] > 0 and 0.0 < pr["call_rate_vs_pattern"] <= 1.5


def test_packed_placement_and_split_mode_lines():
    d = _bench("--workload", "tiny_m4_p1m_f32", "--steps", "3", "--warmup", "1", "--copy-gb", "0.05",
               "--no-cpu-baseline", "--placement", "packed")
    assert d["config"]["placement"] == "packed" and d["roofline"]["timed_launches"] == 3
    s = _bench("--mode", "split", "--workload", "tiny_m4_p1m_f32", "--steps", "3", "--warmup", "1",
               "--no-cpu-baseline")
    assert s["mode"] == "split" and s["blocking_ms"] > 0 and s["mix1_ms"] > 0 and s["round_ms_median"] > 0
    assert s["bytes"]["mix1"] == 4 * (1 << 20) * 2 * 4                # read theta_prev, write x
    assert s["bytes"]["blocking"] == 4 * (1 << 20) * (4 * 4 + 8 + 4)  # with the write-back into theta_local
    assert s["config"]["placement"].startswith("momentum one physical-memory range")
    assert s["unit"] == "GB/s" and s["value"] == s["roofline"]["achieved"] > 0
    assert s["roofline"]["bound"] == "hbm" and s["roofline"]["bytes_per_launch"] == s["bytes"]["blocking"]
