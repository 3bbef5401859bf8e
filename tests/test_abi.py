"""CPU tests of the C ABI: the library loads, exports every entry point the
header declares, validates topologies, and computes the effective mixing
weights bit for bit like the oracle.  No compute call needs a GPU here
(engines are created host-only, device = -1).
"""

import ctypes
import os
import re
import subprocess

import numpy as np
import pytest

import oracle
import paper_2606_22768_amd as fgd
from synth import graphs

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    with open(os.path.join(ROOT, "include", "fgd.h")) as f:
        text = f.read()
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(fgd_\w+)\s*\(", text, re.M)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for required in ["fgd_create", "fgd_set_topology", "fgd_outer_step", "fgd_consensus_distance", "fgd_destroy"]:
        assert required in names


def test_library_exports_every_declared_symbol():
    out = subprocess.run(["nm", "-D", "--defined-only", fgd.LIB_PATH], capture_output=True, text=True, check=True)
    exported = set(re.findall(r"\bT (fgd_\w+)", out.stdout))
    missing = [n for n in declared_functions() if n not in exported]
    assert not missing, f"declared but not exported: {missing}"
    for n in declared_functions():
        assert hasattr(fgd.lib, n)


def test_status_strings():
    assert fgd.fgd_status_string(0) == "FGD_OK"
    assert fgd.fgd_status_string(2) == "FGD_ERR_TOPOLOGY"
    assert fgd.fgd_status_string(99) == "FGD_UNKNOWN_STATUS"


def _random_cases():
    cases = []
    for seed in range(40):
        rng = np.random.default_rng(seed)
        M = int(rng.integers(1, 17))
        rp, ci = graphs.random_symmetric_structure(M, float(rng.uniform(0.1, 0.9)), seed)
        mask = graphs.edge_drop_masks(rp, ci, 1, float(rng.uniform(0, 0.6)), seed)[0]
        w = oracle.round_weights(rp, ci, None, None, "metropolis")  # a doubly-stochastic base W
        cases.append((M, rp, ci, w, mask))
    return cases


@pytest.mark.parametrize("reweight", ["metropolis", "self"])
def test_effective_weights_bit_exact_vs_oracle(reweight):
    """Library and oracle implement the reweighting rules independently; the
    float32 results must agree bit for bit."""
    for M, rp, ci, w, mask in _random_cases():
        a = fgd.fgd_effective_weights(M, rp, ci, w, mask, reweight)
        b = oracle.round_weights(rp, ci, w, mask, reweight)
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32)), (M, reweight)


def test_effective_weights_golden_cases():
    import json
    from fractions import Fraction

    with open(os.path.join(ROOT, "tests", "golden", "metropolis_cases.json")) as f:
        cases = json.load(f)["cases"]
    for c in cases:
        rp, ci = graphs._csr_from_rows(c["rows"])
        mask = graphs.masks_from_live_edges(rp, ci, [c["live"]])[0]
        out = fgd.fgd_effective_weights(c["M"], rp, ci, None, mask, "metropolis")
        for i in range(c["M"]):
            for e in range(rp[i], rp[i + 1]):
                assert out[e] == np.float32(float(Fraction(c["weights"][f"{i},{ci[e]}"]))), c["name"]


def test_engine_rounds_match_oracle_and_upload_tables():
    """A host-only engine stores per-round weights identical to the oracle's."""
    M = 8
    rp, ci = graphs.ring(M)
    masks = graphs.edge_drop_masks(rp, ci, 3, 0.3, seed=5)
    eng = fgd.Engine(M, 100, 104, "f32", device=-1)
    eng.set_topology("mix2", "csr", rp, ci, None, 3, masks, "metropolis")
    eng.set_topology("mix1", "global")
    assert eng.num_cd_rows() == (3 + 1) + (1 + 1) + 1
    for k in range(3):
        a = eng.effective_weights("mix2", k)
        b = oracle.round_weights(rp, ci, None, masks[k], "metropolis")
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32))
    assert eng.min_bytes_per_step() == M * 100 * 20
    eng.close()


def test_host_only_engine_refuses_compute():
    eng = fgd.Engine(4, 64, 64, "bf16", device=-1)
    eng.set_topology("mix1", "global")
    eng.set_topology("mix2", "identity")
    assert eng.min_bytes_per_step() == 4 * 64 * 14
    with pytest.raises(fgd.FgdError) as e:
        fgd.fgd_outer_step(eng.handle, 256, 512, 1024, None, 0)
    assert e.value.status == fgd.FGD_ERR_STATE
    eng.close()


@pytest.mark.parametrize("bad", ["decreasing", "unsorted", "no_diag", "out_of_range", "masked_diag",
                                 "asym_mask", "mask_value", "masks_without_reweight", "not_doubly_stochastic",
                                 "metropolis_directed", "negative_weight", "too_many_rounds", "no_weights"])
def test_topology_rejections(bad):
    M = 5
    rp, ci, w = graphs.ring_weights(M)
    rp, ci, w = rp.copy(), ci.copy(), w.copy()
    masks, reweight, rounds = None, "none", 1
    status = fgd.FGD_ERR_TOPOLOGY
    if bad == "decreasing":
        rp[2] = rp[3] + 1
    elif bad == "unsorted":
        ci[0], ci[1] = ci[1], ci[0]
    elif bad == "no_diag":
        rp, ci = graphs._csr_from_rows([[1, 4], [0, 1, 2], [1, 2, 3], [2, 3, 4], [0, 3, 4]])
        w = np.full(len(ci), 0.5, np.float32)
    elif bad == "out_of_range":
        ci[-1] = M
    elif bad == "masked_diag":
        masks = np.ones((1, len(ci)), np.uint8)
        masks[0, list(ci[rp[0]:rp[1]]).index(0)] = 0
        reweight = "metropolis"
    elif bad == "asym_mask":
        masks = np.ones((1, len(ci)), np.uint8)
        masks[0, rp[0] + list(ci[rp[0]:rp[1]]).index(1)] = 0  # (0,1) dropped but (1,0) live
        reweight = "metropolis"
    elif bad == "mask_value":
        masks = np.full((1, len(ci)), 2, np.uint8)
        reweight = "metropolis"
    elif bad == "masks_without_reweight":
        masks = graphs.edge_drop_masks(rp, ci, 1, 0.9, seed=0)
    elif bad == "not_doubly_stochastic":
        w[0] = 0.9
    elif bad == "metropolis_directed":
        rp, ci = graphs.exponential(M, hops=(1,))
        w, reweight = None, "metropolis"
    elif bad == "negative_weight":
        w[1] = -w[1]
    elif bad == "too_many_rounds":
        rounds, status = fgd.FGD_MAX_ROUNDS + 1, fgd.FGD_ERR_INVALID_ARG
    elif bad == "no_weights":
        w, status = None, fgd.FGD_ERR_INVALID_ARG
    eng = fgd.Engine(M, 16, 16, "f32", device=-1)
    with pytest.raises(fgd.FgdError) as e:
        eng.set_topology("mix2", "csr", rp, ci, w, rounds, masks, reweight)
    assert e.value.status == status, (bad, str(e.value))
    assert fgd.fgd_last_error()
    eng.close()


def test_directed_doubly_stochastic_graph_is_accepted():
    """The directed exponential graph is doubly stochastic but not symmetric;
    it is accepted with its given weights."""
    rp, ci, w = graphs.exponential_weights(16)
    eng = fgd.Engine(16, 16, 16, "f32", device=-1)
    eng.set_topology("mix2", "csr", rp, ci, w, 2)
    assert np.array_equal(eng.effective_weights("mix2", 1), w)
    eng.close()


@pytest.mark.parametrize("field,value", [("num_workers", 0), ("num_workers", 65), ("num_params", -1),
                                         ("ld", 10), ("param_dtype", 7), ("ld", 102)])
def test_create_rejections(field, value):
    kw = dict(num_workers=4, num_params=100, ld=104, param_dtype="f32", device=-1)
    kw[field] = value
    with pytest.raises(fgd.FgdError) as e:
        fgd.fgd_create(**kw)
    assert e.value.status == fgd.FGD_ERR_INVALID_ARG


def test_zero_rounds_is_identity():
    rp, ci, w = graphs.ring_weights(6)
    eng = fgd.Engine(6, 8, 8, "f32", device=-1)
    eng.set_topology("mix1", "csr", rp, ci, w, 0)
    eng.set_topology("mix2", "global")
    assert eng.num_cd_rows() == 2 + 1 + 1
    eng.close()


@pytest.mark.parametrize("field,value,status", [
    ("nesterov", 2, "FGD_ERR_INVALID_ARG"),
    ("nesterov", -1, "FGD_ERR_INVALID_ARG"),
    ("mix1_state", 3, "FGD_ERR_INVALID_ARG"),
    ("state_dtype", 7, "FGD_ERR_INVALID_ARG"),
    ("state_dtype", "bf16", "FGD_ERR_UNSUPPORTED"),  # momentum is float32 only
])
def test_create_rejects_variant_fields(field, value, status):
    kw = dict(num_workers=4, num_params=100, ld=104, param_dtype="f32", device=-1)
    kw[field] = value
    with pytest.raises(fgd.FgdError) as e:
        fgd.fgd_create(**kw)
    assert e.value.status == getattr(fgd, status)


def test_create_rejects_nonzero_reserved_and_wrong_size():
    for size, reserved in ((ctypes.sizeof(fgd.fgd_config), 1), (ctypes.sizeof(fgd.fgd_config) - 8, 0)):
        cfg = fgd.fgd_config(size, 4, 100, 104, fgd.FGD_F32, fgd.FGD_F32, 0.7, 0.9, 1, -1, 0, reserved)
        h = ctypes.c_void_p()
        assert fgd.lib.fgd_create(ctypes.byref(cfg), ctypes.byref(h)) == fgd.FGD_ERR_INVALID_ARG
        assert not h.value


def test_create_accepts_variants_host_only():
    for nesterov in (0, 1):
        for state in (0, 1):
            h = fgd.fgd_create(4, 100, 104, "bf16", device=-1, nesterov=nesterov, mix1_state=state)
            fgd.fgd_destroy(h)


@pytest.mark.parametrize("segs", [
    [(5, 5)],                # empty
    [(10, 20), (15, 30)],    # overlapping
    [(30, 40), (10, 20)],    # descending
    [(0, 101)],              # beyond P
    [(-1, 3)],               # negative
])
def test_subset_rejections(segs):
    eng = fgd.Engine(4, 100, 104, "f32", device=-1)
    try:
        with pytest.raises(fgd.FgdError) as e:
            eng.set_mix2_subset(segs)
        assert e.value.status == fgd.FGD_ERR_INVALID_ARG
    finally:
        eng.close()


def test_subset_limits():
    eng = fgd.Engine(4, 1 << 20, 1 << 20, "f32", device=-1)
    try:
        n = fgd.FGD_MAX_SUBSET_SEGMENTS
        ok = np.stack([np.arange(n) * 4, np.arange(n) * 4 + 2], axis=1)
        eng.set_mix2_subset(ok)                     # the maximum count
        eng.set_mix2_subset([(0, 1), (1, 2)])       # touching segments
        eng.set_mix2_subset(None)                   # cleared
        eng.set_mix2_subset([])
        too_many = np.stack([np.arange(n + 1) * 4, np.arange(n + 1) * 4 + 2], axis=1)
        with pytest.raises(fgd.FgdError) as e:
            eng.set_mix2_subset(too_many)
        assert e.value.status == fgd.FGD_ERR_INVALID_ARG
        assert fgd.lib.fgd_set_mix2_subset(eng.handle, None, 2) == fgd.FGD_ERR_INVALID_ARG
        assert fgd.lib.fgd_set_mix2_subset(eng.handle, None, -1) == fgd.FGD_ERR_INVALID_ARG
    finally:
        eng.close()


MiB2, GiB = 2 << 20, 1 << 30


@pytest.mark.parametrize("M,P,ld,dtype", [(8, 1_100_000_000, 1_100_000_000, "bf16"), (64, 124_000_000, 124_000_000, "f32"),
                                          (16, 500_000_000, 500_000_000, "f32"), (4, 1000, 1000, "f32"),
                                          (3, 8, 8, "bf16")])
@pytest.mark.parametrize("with_x", [False, True])
def test_state_layout_arithmetic(M, P, ld, dtype, with_x):
    """fgd_state_layout: 2 MiB-aligned, non-overlapping [M][ld] arrays in the
    documented order; spread puts the momentum at range_bytes whenever the
    parameter arrays end within it, else packed."""
    es = 2 if dtype == "bf16" else 4
    eng = fgd.Engine(M, P, ld, dtype, device=-1)
    try:
        tb, vb = M * ld * es, M * ld * 4
        up = lambda b: -(-b // MiB2) * MiB2
        packed, ptotal = eng.state_layout(spread=False, with_x=with_x)
        want = [0, up(tb), 2 * up(tb) if with_x else -1, (3 if with_x else 2) * up(tb)]
        assert list(packed) == want
        assert ptotal == want[3] + vb
        for rng in (96 * GiB, 4 * MiB2, 2 * MiB2):
            offs, total = eng.state_layout(spread=True, with_x=with_x, range_bytes=rng)
            assert offs[:3] == packed[:3]
            end = want[3]
            assert offs[3] == (rng if rng >= end else end)
            block = -(-(rng // 3 * 4) // MiB2) * MiB2   # 4/3 of a range, whole 2 MiB pages
            if offs[3] == rng and offs[3] + vb < block:
                assert total == block                    # rounded up to one aligned block
            else:
                assert total == offs[3] + vb
            spans = [(o, o + n) for o, n in zip(offs, (tb, tb, tb, vb)) if o >= 0]
            for o, _ in spans:
                assert o % MiB2 == 0
            spans.sort()
            assert all(a[1] <= b[0] for a, b in zip(spans, spans[1:]))
            assert spans[-1][1] <= total
        # spread = False ignores range_bytes
        assert eng.state_layout(spread=False, with_x=with_x, range_bytes=96 * GiB) == (packed, ptotal)
    finally:
        eng.close()


def test_state_layout_rejections():
    eng = fgd.Engine(8, 1000, 1000, "f32", device=-1)
    try:
        offs, total = (ctypes.c_int64 * 4)(), ctypes.c_int64()
        # a host-only engine cannot derive the range from a device
        assert fgd.lib.fgd_state_layout(eng.handle, 1, 0, 0, offs, ctypes.byref(total)) == fgd.FGD_ERR_STATE
        # packed needs no device
        assert fgd.lib.fgd_state_layout(eng.handle, 0, 0, 0, offs, ctypes.byref(total)) == fgd.FGD_OK
        for spread, wx, rng in ((2, 0, 0), (0, 2, 0), (1, 0, -MiB2), (1, 0, MiB2 + 16), (1, 0, 1 << 20)):
            assert fgd.lib.fgd_state_layout(eng.handle, spread, wx, rng, offs, ctypes.byref(total)) == \
                fgd.FGD_ERR_INVALID_ARG, (spread, wx, rng)
        assert fgd.lib.fgd_state_layout(eng.handle, 0, 0, 0, None, ctypes.byref(total)) == fgd.FGD_ERR_INVALID_ARG
        assert fgd.lib.fgd_state_layout(eng.handle, 0, 0, 0, offs, None) == fgd.FGD_ERR_INVALID_ARG
        assert fgd.lib.fgd_state_layout(None, 0, 0, 0, offs, ctypes.byref(total)) == fgd.FGD_ERR_INVALID_ARG
    finally:
        eng.close()


def test_header_compiles_as_c99_and_links(tmp_path):
    """include/fgd.h is a plain C header: a C99 program that includes it,
    links libfgd.so and calls host-only entry points (a host-only engine and
    the stand-alone weight computation) builds with -Wall -Werror -pedantic
    and runs.  No GPU is touched."""
    src = tmp_path / "abi_check.c"
    src.write_text(r"""
#include <stdio.h>
#include <string.h>
#include "fgd.h"
int main(void) {
    fgd_config c;
    fgd_engine *e = NULL;
    int32_t rp[4] = {0, 2, 5, 7}, ci[7] = {0, 1, 0, 1, 2, 1, 2};
    float w[7], out[7];
    int32_t rows = 0;
    memset(&c, 0, sizeof c);
    c.struct_size = sizeof c;
    c.num_workers = 3;
    c.num_params = 64;
    c.ld = 64;
    c.param_dtype = FGD_F32;
    c.state_dtype = FGD_F32;
    c.outer_lr = 0.7f;
    c.momentum = 0.9f;
    c.nesterov = 1;
    c.device = -1;
    if (fgd_create(&c, &e) != FGD_OK) { printf("create: %s\n", fgd_last_error()); return 1; }
    if (fgd_set_topology(e, FGD_MIX1, FGD_W_GLOBAL_MEAN, NULL, NULL, NULL, 1, NULL, FGD_REWEIGHT_NONE) != FGD_OK) return 2;
    if (fgd_set_topology(e, FGD_MIX2, FGD_W_CSR, rp, ci, NULL, 2, NULL, FGD_REWEIGHT_METROPOLIS) != FGD_OK) return 3;
    if (fgd_num_cd_rows(e, &rows) != FGD_OK || rows != 2 + 1 + 1 + 1 + 1) return 4;
    if (fgd_get_effective_weights(e, FGD_MIX2, 1, w) != FGD_OK) return 5;
    if (fgd_effective_weights(3, rp, ci, NULL, NULL, FGD_REWEIGHT_METROPOLIS, out) != FGD_OK) return 6;
    if (memcmp(w, out, sizeof w) != 0) return 7;
    if (fgd_outer_step(e, NULL, NULL, NULL, NULL, NULL) != FGD_ERR_STATE) return 8;  /* host-only engine */
    if (strcmp(fgd_status_string(FGD_ERR_TOPOLOGY), "FGD_ERR_TOPOLOGY") != 0) return 9;
    fgd_destroy(e);
    printf("ok %g %g %g\n", w[0], w[1], w[2]);
    return 0;
}
""")
    exe = tmp_path / "abi_check"
    inc = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include")
    libdir = os.path.dirname(fgd.LIB_PATH)
    subprocess.run(["gcc", "-std=c99", "-Wall", "-Wextra", "-Werror", "-pedantic", "-I", inc, str(src), "-o", str(exe),
                    "-L", libdir, "-lfgd", f"-Wl,-rpath,{libdir}"], check=True)
    r = subprocess.run([str(exe)], capture_output=True, text=True)
    assert r.returncode == 0, (r.returncode, r.stdout, r.stderr)
    # Path graph 0-1-2, Metropolis: degrees 1, 2, 1 -> w01 = w12 = 1/3, w00 = w22 = 2/3, w11 = 1/3.
    assert r.stdout.split()[:4] == ["ok", f"{np.float32(2 / 3):g}", f"{np.float32(1 / 3):g}", f"{np.float32(1 / 3):g}"]


def test_binding_refuses_to_import_without_the_library(tmp_path):
    """No fallback: a copy of the package without libfgd.so fails to import,
    naming the missing library, rather than running anything on the CPU."""
    import shutil
    pkg = os.path.join(ROOT, "paper_2606_22768_amd")
    dst = tmp_path / "paper_2606_22768_amd"
    dst.mkdir()
    for name in os.listdir(pkg):
        if name.endswith(".py"):
            shutil.copy(os.path.join(pkg, name), dst / name)
    assert not (dst / "libfgd.so").exists()
    code = ("import sys; sys.path.insert(0, sys.argv[1])\n"
            "try:\n    import paper_2606_22768_amd\nexcept ImportError as e:\n    print('refused:', e); sys.exit(3)\n"
            "sys.exit(0)\n")
    r = subprocess.run(["python", "-c", code, str(tmp_path)], capture_output=True, text=True, cwd=str(tmp_path))
    assert r.returncode == 3, (r.returncode, r.stdout, r.stderr)
    assert "libfgd.so is missing" in r.stdout


def _tree_copy(tmp_path, with_lib):
    """A copy of the package (sources, binding, optionally the built library and
    its sidecar) and the header under tmp_path."""
    import shutil
    pkg = os.path.join(ROOT, "paper_2606_22768_amd")
    dst = tmp_path / "paper_2606_22768_amd"
    shutil.copytree(os.path.join(pkg, "csrc"), dst / "csrc")
    for name in os.listdir(pkg):
        if name.endswith(".py") or (with_lib and name in ("libfgd.so", "libfgd.so.json")):
            shutil.copy(os.path.join(pkg, name), dst / name)
    (tmp_path / "include").mkdir()
    shutil.copy(os.path.join(ROOT, "include", "fgd.h"), tmp_path / "include" / "fgd.h")
    return dst


def test_library_carries_the_hashes_of_its_sources():
    from paper_2606_22768_amd import build
    want = build.source_hashes()
    assert fgd.library_source_hash() == want
    assert build.read_sidecar() == want
    assert not build.needs_build()


def test_stale_library_is_rebuilt_or_refused(tmp_path):
    """Editing a kernel source in a copy of the tree marks the copied library
    stale for ensure_built (which then rebuilds) and makes the binding refuse
    to load it; the unedited copy is accepted."""
    from paper_2606_22768_amd import build
    dst = _tree_copy(tmp_path, with_lib=True)
    lib = str(dst / "libfgd.so")
    assert not build.needs_build(lib, str(tmp_path))
    code = ("import sys; sys.path.insert(0, sys.argv[1])\n"
            "try:\n    import paper_2606_22768_amd\nexcept ImportError as e:\n    print('refused:', e); sys.exit(3)\n"
            "print('loaded'); sys.exit(0)\n")
    r = subprocess.run(["python", "-c", code, str(tmp_path)], capture_output=True, text=True, cwd=str(tmp_path))
    assert r.returncode == 0 and "loaded" in r.stdout, (r.stdout, r.stderr)
    with open(dst / "csrc" / "kernels.hpp", "a") as f:
        f.write("\n// edited\n")
    assert build.needs_build(lib, str(tmp_path))
    assert build.source_hashes(str(tmp_path))["step"] != build.source_hashes()["step"]
    r = subprocess.run(["python", "-c", code, str(tmp_path)], capture_output=True, text=True, cwd=str(tmp_path))
    assert r.returncode == 3, (r.returncode, r.stdout, r.stderr)
    assert "built from other sources" in r.stdout
    os.remove(dst / "libfgd.so.json")
    with open(dst / "csrc" / "kernels.hpp", "rb") as f:
        text = f.read()
    with open(dst / "csrc" / "kernels.hpp", "wb") as f:
        f.write(text.replace(b"\n// edited\n", b""))
    assert build.needs_build(lib, str(tmp_path))  # no record of what it was built from


@pytest.mark.parametrize("call", ["outer_step", "mix1", "outer_step_blocking", "consensus_distance"])
def test_consensus_outputs_are_checked_before_any_launch(call):
    """The kernels write rows x M doubles through the raw cd_out / out pointer,
    so the wrapper refuses a buffer of another dtype, a smaller one, a
    non-contiguous one or one off the engine's device before calling the C
    ABI (a host-only engine: any call that got through would fail there)."""
    import torch
    M, P = 8, 64
    eng = fgd.Engine(M, P, P, "f32", device=-1)
    eng.set_topology("mix1", "global")
    rp, ci, w = graphs.ring_weights(M)
    eng.set_topology("mix2", "csr", rp, ci, w, rounds=2)
    rows = {"outer_step": eng.num_cd_rows(), "mix1": eng.num_cd_rows_split()[0],
            "outer_step_blocking": eng.num_cd_rows_split()[1], "consensus_distance": 1}[call]
    a = torch.zeros((M, P))

    def run(out):
        if call == "outer_step":
            eng.outer_step(a, a, a, out)
        elif call == "mix1":
            eng.mix1(a, a, None, out)
        elif call == "outer_step_blocking":
            eng.outer_step_blocking(a, a, a, a, out)
        else:
            eng.consensus_distance(a, out)

    with pytest.raises(TypeError, match="float64"):
        run(torch.zeros(rows * M, dtype=torch.float32))
    with pytest.raises(ValueError, match="needs at least"):
        run(torch.zeros(rows * M - 1, dtype=torch.float64))
    with pytest.raises(ValueError, match="contiguous"):
        run(torch.zeros((M, 2 * rows), dtype=torch.float64)[:, ::2])
    with pytest.raises(ValueError, match="cuda"):
        run(torch.zeros((rows, M), dtype=torch.float64))
    eng.close()


@pytest.mark.parametrize("dtype", [None, "bf16"])
def test_js_buffers_are_checked_before_any_launch(dtype):
    """js_distance writes d, the means, the token sets and its workspace
    through raw pointers, so a caller's buffer of another dtype, a smaller
    one or a non-contiguous one is refused before anything is enqueued, and
    so are tensors off the GPU (host tensors here: any call that got through
    the checks would stop at the last one)."""
    import torch
    M, U, K, k = 3, 5, 64, 10
    t = torch.float32 if dtype is None else torch.bfloat16
    A, W = torch.zeros((U, K), dtype=t), torch.zeros((M, U, K), dtype=t)
    ws = fgd.fgd_js_workspace_size("f32" if dtype is None else dtype, M, U)

    def run(**kw):
        fgd.js_distance(A, W, top_k=k, **kw)

    with pytest.raises(TypeError, match="float64"):
        run(d_out=torch.zeros((M, U), dtype=torch.float32))
    with pytest.raises(ValueError, match="needs at least"):
        run(d_out=torch.zeros(M * U - 1, dtype=torch.float64))
    with pytest.raises(ValueError, match="contiguous"):
        run(d_out=torch.zeros((M, 2 * U), dtype=torch.float64)[:, ::2])
    with pytest.raises(ValueError, match="needs at least"):
        run(mean_out=torch.zeros(M - 1, dtype=torch.float64))
    with pytest.raises(TypeError, match="int32"):
        run(topk_out=torch.zeros((U, k), dtype=torch.int64))
    with pytest.raises(ValueError, match="needs at least"):
        run(topk_out=torch.zeros((U, k - 1), dtype=torch.int32))
    with pytest.raises(ValueError, match="needs at least"):
        run(workspace=torch.zeros(ws - 1, dtype=torch.uint8))
    with pytest.raises(ValueError, match="GPU"):
        run(workspace=torch.zeros(ws, dtype=torch.uint8))


def test_noalloc_consensus_rejects_arguments_before_any_device_call():
    """The scratch-free consensus call checks its arguments first: more workers
    than its static scratch holds, bad sizes, dtype or alignment."""
    L = fgd.lib
    assert L.fgd_consensus_distance_noalloc(65, 16, 16, 0, 256, 256, None) == fgd.FGD_ERR_INVALID_ARG
    assert "num_workers 65" in fgd.fgd_last_error()
    assert L.fgd_consensus_distance_noalloc(0, 16, 16, 0, 256, 256, None) == fgd.FGD_ERR_INVALID_ARG
    assert L.fgd_consensus_distance_noalloc(4, 17, 16, 0, 256, 256, None) == fgd.FGD_ERR_INVALID_ARG
    assert L.fgd_consensus_distance_noalloc(4, 16, 16, 7, 256, 256, None) == fgd.FGD_ERR_INVALID_ARG
    assert L.fgd_consensus_distance_noalloc(4, 16, 16, 0, 264, 256, None) == fgd.FGD_ERR_INVALID_ARG
    assert L.fgd_consensus_distance_noalloc(4, 16, 16, 0, 256, 260, None) == fgd.FGD_ERR_INVALID_ARG
    assert L.fgd_consensus_distance_noalloc(4, 6, 6, 0, 256, 256, None) == fgd.FGD_ERR_INVALID_ARG  # 24-byte rows


def _variant(M, t1, t2, dtype="f32", subset=None, mix1_state=False, P=4096):
    from tests import _parity as pa
    eng = fgd.Engine(M, P, P, dtype, device=-1, mix1_state=mix1_state)
    eng.set_topology_dict("mix1", t1)
    eng.set_topology_dict("mix2", t2)
    if subset:
        eng.set_mix2_subset(subset)
    v = eng.step_variant()
    eng.close()
    return v


def test_step_variant_choice():
    """The worker-group kernel serves 64 workers on sparse CSR tables within
    its round and LDS limits; everything else runs on the lane-per-parameter
    kernel."""
    from tests import _parity as pa
    reg4, ring = ("regular", "metropolis", 4), ("ring", "metropolis", 0.1)
    G = ("global",)
    wg, lpp = "worker-groups", "lane-per-param"
    assert _variant(64, pa.topo(reg4, 64, 1), pa.topo(reg4, 64, 3)) == wg            # LocalM1M2, 64 x 124M shape
    assert _variant(64, pa.topo(reg4, 64, 1), pa.topo(reg4, 64, 3), "bf16") == wg
    assert _variant(64, pa.topo(G, 64, 1), pa.topo(ring, 64, 4)) == wg               # GlobalM1LocalM2
    assert _variant(64, pa.topo(reg4, 64, 2), pa.topo(reg4, 64, 4)) == wg            # the unrolled maxima
    assert _variant(64, pa.topo(reg4, 64, 3), pa.topo(reg4, 64, 1)) == lpp           # Mix1 rounds beyond 2
    assert _variant(64, pa.topo(reg4, 64, 1), pa.topo(reg4, 64, 5)) == lpp           # Mix2 rounds beyond 4
    assert _variant(64, pa.topo(G, 64, 1), pa.topo(("complete",), 64, 1)) == lpp     # 64-entry rows
    assert _variant(64, pa.topo(("identity",), 64, 0), pa.topo(reg4, 64, 1)) == lpp  # identity Mix1
    assert _variant(64, pa.topo(G, 64, 1), pa.topo(G, 64, 1)) == lpp                 # no CSR Mix2
    assert _variant(64, pa.topo(G, 64, 1), pa.topo(reg4, 64, 1), subset=[(0, 100)]) == lpp
    assert _variant(64, pa.topo(G, 64, 1), pa.topo(reg4, 64, 1), mix1_state=True) == lpp
    assert _variant(32, pa.topo(reg4, 32, 1), pa.topo(reg4, 32, 3)) == lpp
    assert _variant(63, pa.topo(G, 63, 1), pa.topo(ring, 63, 1)) == lpp
    # Rows of up to 15 entries are accepted: two rounds of such tables
    # (15 KiB) beside 65 KiB of rows (a padded table adds a zero row per
    # wave) fill the 80 KiB LDS budget of a block exactly; three exceed it.
    dense = ("er_mh", 0.1, 0.0)
    t = pa.topo(dense, 64, 1, seed=3)
    assert np.diff(t["row_ptr"]).max() == 15
    assert _variant(64, pa.topo(dense, 64, 1, seed=3), pa.topo(dense, 64, 1, seed=3)) == wg
    assert _variant(64, pa.topo(dense, 64, 1, seed=3), pa.topo(dense, 64, 2, seed=3)) == lpp
    assert _variant(64, pa.topo(G, 64, 1), pa.topo(dense, 64, 1, seed=3)) == wg
    assert _variant(64, pa.topo(ring, 64, 2), pa.topo(ring, 64, 4)) == wg
