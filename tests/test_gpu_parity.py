"""GPU parity: the HIP engine against the CPU oracle, element by element, on
seeded inputs that span several tiles and end in a ragged tail, over worker
counts, storage types, mixing kinds, rounds, masks and reweighting rules.
Every call goes through the C ABI (libfgd.so).
"""

import numpy as np
import pytest

import oracle
from synth import configs, tensors
from tests import _parity as pa

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def env():
    import torch

    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    import paper_2606_22768_amd as fgd

    return fgd, torch


G, ID = ("global",), ("identity",)
RING, EXP = ("ring", "given"), ("exp", "given")
RING_MH = ("ring", "metropolis", 0.1)
REG4 = ("regular", "metropolis", 4)

# (M, P, dtype, mix1 spec, K1, mix2 spec, K2, ld)
CASES = [
    (8, 3079, "f32", G, 1, RING, 1, None),                        # GlobalM1LocalM2, ring
    (8, 3079, "bf16", G, 1, RING_MH, 1, None),                    # bf16, per-round drops + Metropolis
    (16, 3079, "f32", G, 1, EXP, 2, None),                        # directed exponential graph, 2 rounds
    (64, 775, "f32", REG4, 1, REG4, 3, None),                     # 4-regular Metropolis, 1 + 3 rounds
    (64, 775, "bf16", REG4, 1, REG4, 3, None),
    (4, 3079, "f32", RING, 2, RING, 1, 3088),                     # ld > P
    (8, 3079, "f32", ("matching",), 1, ("matching",), 1, None),   # LocalM1M2 (pairwise gossip)
    (8, 3079, "f32", ID, 0, G, 1, None),                          # DiLoCo
    (8, 3079, "bf16", G, 1, ID, 0, None),                         # GlobalM1
    (5, 2051, "f32", ("er_mh", 0.6, 0.2), 2, ("ring_self", 0.3), 3, None),  # M not a power of two
    (3, 1001, "bf16", ("complete",), 1, G, 1, None),
    (1, 999, "f32", G, 1, ID, 0, None),
    (1, 1003, "bf16", ID, 0, ("complete",), 2, None),
    (12, 2000, "f32", ("er_mh", 0.4, 0.1), 1, ("er_mh", 0.4, 0.1), 2, None),
    (33, 700, "f32", ("er_mh", 0.2, 0.1), 1, ("er_mh", 0.2, 0.1), 1, None),
    (32, 900, "bf16", ("er_mh", 0.2, 0.1), 2, G, 1, None),        # kinds chosen at run time
    (2, 17, "f32", G, 1, ("complete",), 1, None),
    (16, 5, "bf16", G, 1, EXP, 1, 8),                             # P smaller than one vector
    (7, 4099, "bf16", ("ring_self", 0.2), 1, ("er_mh", 0.5, 0.3), 2, 4104),
    # The largest worker count with the most rounds in both slots: the most LDS rows and consensus rows (19).
    (64, 600, "f32", REG4, 8, REG4, 8, None),
    (64, 520, "bf16", ("er_mh", 0.1, 0.2), 8, ("ring_self", 0.3), 8, None),   # padded tables at 8 rounds
    (48, 777, "f32", ("er_mh", 0.2, 0.1), 8, G, 1, None),
]


def _id(c):
    return f"M{c[0]}-P{c[1]}-{c[2]}-{c[3][0]}{c[4]}-{c[5][0]}{c[6]}" + (f"-ld{c[7]}" if c[7] else "")


@pytest.mark.parametrize("case", CASES, ids=_id)
def test_step_parity(env, case):
    fgd, torch = env
    M, P, dtype, s1, k1, s2, k2, ld = case
    print(f"[parity] {_id(case)}", flush=True)
    pa.run_case(fgd, torch, M, P, dtype, s1, k1, s2, k2, ld=ld, seed=M + P)


# 32 and 64 workers (one or two parameters per lane, every worker's rows in
# the lane's registers) with the kinds of the paper's configurations: ragged
# tails, P below one tile, ld > P, padded tables.
LARGE_M_CASES = [
    (64, 3 * 4096 + 37, "f32", G, 1, REG4, 3, None),               # GlobalM1LocalM2
    (64, 1000, "bf16", REG4, 1, REG4, 3, 1016),                    # LocalM1M2, ld > P
    (64, 63, "f32", REG4, 1, REG4, 1, None),                       # P below one tile
    (64, 640, "bf16", ("er_mh", 0.2, 0.3), 2, ("er_mh", 0.2, 0.3), 3, None),  # padded tables, exact tiles
    (64, 333, "f32", ID, 0, G, 1, None),                           # DiLoCo
    (32, 2049, "f32", G, 1, ("er_mh", 0.3, 0.2), 2, None),
    (32, 130, "bf16", G, 1, ID, 0, None),                          # GlobalM1
    (32, 4100, "bf16", ("ring_self", 0.2), 2, ("er_mh", 0.4, 0.1), 1, 4104),
    # Dense W (64 and about 40 entries per row): sums long enough that one
    # float32 chain per row would approach the 1e-6 bar on their small means.
    (64, 2661, "f32", ("complete",), 2, G, 1, None),
    (48, 1777, "f32", ("er_mh", 0.9, 0.1), 3, ("complete",), 2, None),
    (64, 901, "bf16", ("complete",), 1, ("er_mh", 0.7, 0.0), 2, None),
]


@pytest.mark.parametrize("case", LARGE_M_CASES, ids=_id)
def test_large_m_step_parity(env, case):
    fgd, torch = env
    M, P, dtype, s1, k1, s2, k2, ld = case
    print(f"[parity-large-m] {_id(case)}", flush=True)
    pa.run_case(fgd, torch, M, P, dtype, s1, k1, s2, k2, ld=ld, seed=M * 7 + P)


@pytest.mark.parametrize("nesterov", [True, False])
def test_large_m_step_without_consensus_and_plain_momentum(env, nesterov):
    fgd, torch = env
    print(f"[parity-large-m] nesterov={nesterov} no consensus", flush=True)
    pa.run_case(fgd, torch, 64, 2 * 4096 + 5, "f32", REG4, 1, REG4, 3, with_cd=False, nesterov=nesterov, seed=11)
    pa.run_case(fgd, torch, 32, 1500, "bf16", G, 1, ("er_mh", 0.3, 0.2), 1, nesterov=nesterov, seed=12)


def test_tiny_workload_full(env):
    """The 4-worker, 1,048,576-parameter float32 workload in full (global
    Mix1, ring Mix2, zero momentum)."""
    fgd, torch = env
    w = configs.WORKLOADS["tiny_m4_p1m_f32"]
    print("[parity] tiny_m4_p1m_f32", flush=True)
    pa.run_case(fgd, torch, w["M"], w["P"], w["dtype"], w["mix1"], w["k1"], w["mix2"], w["k2"],
                seed=w["seed"], mom_std=w["mom_std"])


def test_without_consensus(env):
    fgd, torch = env
    pa.run_case(fgd, torch, 8, 3079, "bf16", G, 1, RING_MH, 1, with_cd=False)
    pa.run_case(fgd, torch, 64, 775, "f32", REG4, 1, REG4, 2, with_cd=False)


def test_empty_parameters(env):
    """P = 0: nothing is read or written; every consensus entry is 0."""
    fgd, torch = env
    M = 4
    eng = fgd.Engine(M, 0, 16, "f32", device=0)
    t = pa.topo(RING, M, 1)
    eng.set_topology_dict("mix1", pa.topo(G, M, 1))
    eng.set_topology_dict("mix2", t)
    x = torch.ones((M, 16), device="cuda")
    y = torch.ones((M, 16), device="cuda")
    v = torch.ones((M, 16), device="cuda")
    cd = torch.full((eng.num_cd_rows(), M), 7.0, dtype=torch.float64, device="cuda")
    eng.outer_step(x, y, v, cd)
    torch.cuda.synchronize()
    assert torch.all(x == 1) and torch.all(v == 1) and torch.all(cd == 0)
    eng.close()


def test_deterministic_reruns(env):
    """Two runs on the same inputs are bit-identical, consensus included."""
    fgd, torch = env
    a = pa.run_case(fgd, torch, 8, 5000, "bf16", G, 1, RING_MH, 1, seed=3)
    b = pa.run_case(fgd, torch, 8, 5000, "bf16", G, 1, RING_MH, 1, seed=3)
    for x, y in zip(a, b):
        assert np.array_equal(x, y)


def test_consecutive_steps(env):
    """Three steps in a row on one engine, with new edge masks every step
    (stream-ordered re-uploads of the tables).  The oracle carries the state
    from step to step; before each step the engine's arrays are loaded with
    the oracle's state, so no engine output feeds the oracle."""
    fgd, torch = env
    M, P = 8, 4096 + 13
    ld = pa.aligned_ld(P)
    tp, tl, v = tensors.numpy_inputs(M, P, ld=ld, dtype="bf16", seed=5)
    dev = torch.device("cuda:0")
    g_tp = torch.from_numpy(tp.view(np.int16)).to(dev).view(torch.bfloat16)
    g_tl = torch.from_numpy(tl.view(np.int16)).to(dev).view(torch.bfloat16)
    g_v = torch.from_numpy(v).to(dev)
    eng = fgd.Engine(M, P, ld, "bf16", device=0)
    t1 = pa.topo(G, M, 1)
    eng.set_topology_dict("mix1", t1)
    cur_t, cur_v = tp, v
    for step in range(3):
        t2 = configs.topology(RING_MH, M, 1, seed=0, step=step)
        eng.set_topology_dict("mix2", t2)
        g_tp.copy_(torch.from_numpy(cur_t.view(np.int16)).to(dev).view(torch.bfloat16))
        g_v.copy_(torch.from_numpy(cur_v).to(dev))
        ref_t, ref_v, ref_cd = oracle.outer_step(cur_t, tl, cur_v, oracle.Mix.from_topology(t1),
                                                 oracle.Mix.from_topology(t2), P=P)
        cd = torch.zeros((eng.num_cd_rows(), M), dtype=torch.float64, device=dev)
        eng.outer_step(g_tp, g_tl, g_v, cd)
        torch.cuda.synchronize()
        got_t = g_tp.view(torch.int16).cpu().numpy().view(np.uint16)
        scale = float(np.abs(tensors.bf16_bits_to_f32(cur_t)).max())
        pa.compare_outputs("bf16", got_t, ref_t, g_v.cpu().numpy(), ref_v, P, scale)
        pa.compare_step_cd(cd.cpu().numpy(), ref_cd, ref_t, "bf16", P, scale)
        cur_t, cur_v = ref_t, ref_v
    eng.close()


@pytest.mark.parametrize("M,P,dtype,ld", [(4, 3079, "f32", None), (8, 5003, "bf16", 5008), (16, 1030, "f32", None),
                                          (64, 777, "f32", None), (5, 999, "bf16", None), (1, 64, "f32", None)])
def test_standalone_consensus(env, M, P, dtype, ld):
    """fgd_consensus_distance against the oracle's S_m."""
    fgd, torch = env
    ld = pa.aligned_ld(P) if ld is None else ld
    tp, _, _ = tensors.numpy_inputs(M, ld, dtype=dtype, seed=M)
    ref = oracle.consensus(tp, P=P)
    eng = fgd.Engine(M, P, ld, dtype, device=0)
    x = torch.from_numpy(tp if dtype == "f32" else tp.view(np.int16)).cuda()
    if dtype == "bf16":
        x = x.view(torch.bfloat16)
    out = torch.full((M,), float("nan"), dtype=torch.float64, device="cuda")
    eng.consensus_distance(x, out)
    torch.cuda.synchronize()
    pa.compare_cd(out.cpu().numpy()[None, :], ref[None, :])
    eng.close()


# Sizes large enough that the persistent grid (one block per CU at 16 or
# fewer workers, two at 32 and 64) strides over several tiles per block, so
# the consensus accumulators carry across tiles; every output is compared.
MULTI_TILE_CASES = [
    (8, 600_003, "f32", G, 1, RING_MH, 1),           # ~2.3 tiles per block
    (8, 1_200_001, "bf16", G, 1, RING_MH, 1),        # ~4.6
    (16, 700_001, "f32", G, 1, EXP, 2),              # ~2.7
    (64, 200_003, "f32", REG4, 1, REG4, 3),          # ~1.5 (V = 1, 512 blocks)
    (32, 600_001, "bf16", G, 1, ("er_mh", 0.3, 0.2), 2),  # ~2.3 (V = 2, 512 blocks)
]


@pytest.mark.parametrize("case", MULTI_TILE_CASES, ids=lambda c: f"M{c[0]}-P{c[1]}-{c[2]}")
def test_multi_tile_per_block_parity(env, case):
    fgd, torch = env
    M, P, dtype, s1, k1, s2, k2 = case
    print(f"[parity] multi-tile {case}", flush=True)
    pa.run_case(fgd, torch, M, P, dtype, s1, k1, s2, k2, seed=61)


@pytest.mark.parametrize("i", range(100))
def test_standalone_consensus_random(env, i):
    """fgd_consensus_distance on seeded random shapes and storages: plain
    rows, identical workers (S = 0 in double; float32 means of equal values
    sit at the rounding floor) and one worker offset from the rest."""
    fgd, torch = env
    rng = np.random.default_rng(4000 + i)
    M = int(rng.choice([1, 2, 3, 5, 8, 9, 16, 17, 31, 32, 47, 64]))
    P = int(rng.integers(1, 20000))
    dtype = str(rng.choice(["f32", "bf16"]))
    per = 4 if dtype == "f32" else 8
    ld = (P + int(rng.integers(0, 3)) * per + per - 1) // per * per
    tp, _, _ = tensors.numpy_inputs(M, ld, dtype=dtype, seed=4000 + i)
    kind = int(rng.integers(0, 3))
    if kind == 1:
        tp[:] = tp[:1]
    elif kind == 2 and M > 1:  # all rows equal but one, offset by 0.01
        tp[:] = tp[:1]
        j = int(rng.integers(0, M))
        if dtype == "f32":
            tp[j] = tp[j] + np.float32(0.01)
        else:
            tp[j] = tensors.f32_to_bf16_bits(tensors.bf16_bits_to_f32(tp[j]) + np.float32(0.01))
    print(f"[parity] standalone consensus {i}: M={M} P={P} ld={ld} {dtype} kind={kind}", flush=True)
    ref = oracle.consensus(tp, P=P)
    eng = fgd.Engine(M, P, ld, dtype, device=0)
    x = torch.from_numpy(tp if dtype == "f32" else tp.view(np.int16)).cuda()
    if dtype == "bf16":
        x = x.view(torch.bfloat16)
    out = torch.full((M,), float("nan"), dtype=torch.float64, device="cuda")
    eng.consensus_distance(x, out)
    torch.cuda.synchronize()
    vals = tensors.bf16_bits_to_f32(tp) if dtype == "bf16" else tp
    scale = float(np.abs(vals[:, :P]).max())
    pa.compare_cd(out.cpu().numpy()[None, :], ref[None, :], pa.cd_floor(P, scale))
    eng.close()


def test_fused_theta_row_matches_standalone(env):
    """The fused consensus row of theta' equals the standalone kernel run on
    the stored theta' (two different kernels, same definition)."""
    fgd, torch = env
    M, P = 8, 20000
    _, _, cd = pa.run_case(fgd, torch, M, P, "f32", G, 1, RING, 1, seed=2)
    tp, tl, v = tensors.numpy_inputs(M, P, seed=2)
    t1, t2 = pa.topo(G, M, 1, 2), pa.topo(RING, M, 1, 9)
    out_t, _, _ = pa.run_engine(fgd, torch, M, P, P, "f32", t1, t2, tp, tl, v, with_cd=False)
    eng = fgd.Engine(M, P, P, "f32", device=0)
    out = torch.zeros(M, dtype=torch.float64, device="cuda")
    eng.consensus_distance(torch.from_numpy(out_t).cuda(), out)
    torch.cuda.synchronize()
    np.testing.assert_allclose(out.cpu().numpy(), cd[-1], rtol=1e-9)
    eng.close()


def test_non_default_stream(env):
    """The step runs on a torch stream that is not the null stream: torch and
    the library share one HIP runtime, so the stream handle is valid."""
    fgd, torch = env
    M, P = 8, 5000
    ld = pa.aligned_ld(P)
    tp, tl, v = tensors.numpy_inputs(M, P, ld=ld, seed=21)
    t1, t2 = pa.topo(G, M, 1), pa.topo(RING, M, 1)
    ref_t, ref_v, ref_cd = oracle.outer_step(tp, tl, v, oracle.Mix.from_topology(t1), oracle.Mix.from_topology(t2),
                                             P=P)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        g_tp, g_tl, g_v = (torch.from_numpy(a).cuda() for a in (tp, tl, v))
        eng = fgd.Engine(M, P, ld, "f32", device=0)
        eng.set_topology_dict("mix1", t1)
        eng.set_topology_dict("mix2", t2)
        cd = torch.zeros((eng.num_cd_rows(), M), dtype=torch.float64, device="cuda")
        eng.outer_step(g_tp, g_tl, g_v, cd)
    s.synchronize()
    got_t = g_tp.cpu().numpy()
    pa.compare_outputs("f32", got_t, ref_t, g_v.cpu().numpy(), ref_v, P)
    pa.compare_step_cd(cd.cpu().numpy(), ref_cd, ref_t, "f32", P, float(np.abs(tp).max()))
    eng.close()


def test_abi_errors_on_device(env):
    """Bad calls return an error and launch nothing."""
    fgd, torch = env
    M, P = 4, 1024
    eng = fgd.Engine(M, P, P, "f32", device=0)
    x = torch.zeros((M, P), device="cuda")
    y = torch.zeros((M, P), device="cuda")
    v = torch.zeros((M, P), device="cuda")
    with pytest.raises(fgd.FgdError) as e:
        fgd.fgd_outer_step(eng.handle, x, y, v)
    assert e.value.status == fgd.FGD_ERR_STATE
    eng.set_topology_dict("mix1", pa.topo(G, M, 1))
    eng.set_topology_dict("mix2", pa.topo(RING, M, 1))
    with pytest.raises(fgd.FgdError) as e:
        fgd.fgd_outer_step(eng.handle, x, x, v)  # theta_local aliases theta_prev
    assert e.value.status == fgd.FGD_ERR_INVALID_ARG
    with pytest.raises(fgd.FgdError) as e:
        fgd.fgd_outer_step(eng.handle, x.data_ptr() + 4, y, v)  # misaligned rows
    assert e.value.status == fgd.FGD_ERR_INVALID_ARG
    with pytest.raises(fgd.FgdError) as e:
        fgd.fgd_outer_step(eng.handle, x, y, None)
    assert e.value.status == fgd.FGD_ERR_INVALID_ARG
    torch.cuda.synchronize()
    assert torch.all(x == 0) and torch.all(v == 0)
    eng.close()
