"""GPU parity of split execution (Appendix A, Algorithm 1: Mix1 launched at
the start of a round, the blocking Mix2 and the optimizer at its end)
against the oracle's two halves, through the C ABI.

Each half is checked alone on the same inputs: the Mix1 half's stored x and
consensus rows against the oracle's Mix1 half; the blocking half is fed the
oracle's stored x (uploaded), so its outputs are compared without the
rounding of x in between.  A last test runs both halves on separate streams
with a stand-in inner loop between them, as a round would.
"""

import numpy as np
import pytest

import oracle
from synth import tensors
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

# As many Mix2 subset segments as the engine accepts (4096), one in each cell
# of 3 parameters, lengths 1 to 3, some touching the next.
_rng = np.random.default_rng(5)
DENSE_SEGMENTS = [(3 * i + int(_rng.integers(0, 2)), 3 * i + 3 - int(_rng.integers(0, 2))) for i in range(4096)]

# (M, P, dtype, mix1, K1, mix2, K2, state, subset)
CASES = [
    (8, 3079, "bf16", G, 1, RING_MH, 1, False, None),                 # GlobalM1LocalM2
    (8, 3079, "f32", G, 1, RING, 1, True, None),                      # GlobalM1SLocalM2
    (8, 10007, "bf16", G, 1, RING_MH, 1, True, [(0, 3300), (9000, 10007)]),  # ... -subset
    (16, 3079, "f32", G, 1, EXP, 2, False, None),
    (64, 775, "f32", REG4, 1, REG4, 3, False, None),                  # CSR Mix1 (run-time kinds)
    (64, 775, "bf16", REG4, 1, REG4, 3, True, [(10, 300)]),
    (8, 3079, "f32", ("matching",), 2, ("matching",), 1, True, None),  # LocalM1M2
    (8, 3079, "bf16", ID, 0, G, 1, False, None),                      # DiLoCo
    (5, 2051, "bf16", ("er_mh", 0.6, 0.2), 2, ("ring_self", 0.3), 1, False, [(7, 8), (100, 2000)]),
    (1, 999, "f32", G, 1, ID, 0, True, None),
    # Most rounds at the largest worker count: the Mix1 half's per-chunk partials hold 9 rows, the blocking half 10.
    (64, 600, "f32", REG4, 8, REG4, 8, True, [(0, 128), (300, 600)]),
    (64, 520, "bf16", ("er_mh", 0.1, 0.2), 8, ("ring_self", 0.3), 8, False, None),
    (8, 3 * 4096 + 123, "bf16", G, 1, RING_MH, 1, True, DENSE_SEGMENTS),
    # Enough tiles that the Mix1 half's chunks hold several tiles each and the
    # blocking half's blocks stride over several tiles.
    (8, 4_300_003, "f32", G, 1, RING_MH, 1, False, [(0, 1_420_000), (3_870_000, 4_300_003)]),
]


def _dev_rows(torch, a, dtype):
    t = torch.from_numpy(a.view(np.int16) if dtype == "bf16" else a).cuda()
    return t.view(torch.bfloat16) if dtype == "bf16" else t


def _host_rows(torch, t, dtype):
    return t.view(torch.int16).cpu().numpy().view(np.uint16) if dtype == "bf16" else t.cpu().numpy()


def _ids(c):
    return (f"M{c[0]}-P{c[1]}-{c[2]}-{c[3][0]}{c[4]}-{c[5][0]}{c[6]}-state{int(c[7])}"
            + (f"-subset{len(c[8])}" if c[8] else ""))


@pytest.mark.parametrize("write_local", [False, True], ids=["keep-local", "write-local"])
@pytest.mark.parametrize("case", CASES, ids=_ids)
def test_split_halves(env, case, write_local):
    _split_case(env, case, write_local)


@pytest.mark.parametrize("i", range(200))
def test_split_halves_random_configurations(env, i):
    """The seeded random configurations of the fused-step variants tests
    (worker count, size, storage, Mix kinds and rounds, masks, reweighting,
    optimizer form, state mix, subset) through both halves."""
    from tests.test_gpu_variants import _random_case

    c = _random_case(5000 + i)
    _split_case(env, (c["M"], c["P"], c["dtype"], c["s1"], c["k1"], c["s2"], c["k2"], c["state"], c["subset"]),
                bool(i % 2))


def _split_case(env, case, write_local):
    fgd, torch = env
    M, P, dtype, s1, k1, s2, k2, state, subset = case
    print(f"[split] {case[:8]} subset={None if subset is None else len(subset)} segments "
          f"write_local={write_local}", flush=True)
    ld = pa.aligned_ld(P)
    tp, tl, v = tensors.numpy_inputs(M, P, ld=ld, dtype=dtype, mom_std=1e-3, seed=53)
    t1, t2 = pa.topo(s1, M, k1, 53), pa.topo(s2, M, k2, 60)
    m1, m2 = oracle.Mix.from_topology(t1), oracle.Mix.from_topology(t2)
    ref_x, ref_vm, ref_cd1 = oracle.mix1_split(tp, m1, mom=v, mix1_state=state, P=P)
    v_in = ref_vm if state else v
    ref_t, ref_tl, ref_v, ref_cd2 = oracle.outer_blocking(ref_x, tp, tl, v_in, m2, P=P, subset=subset,
                                                          write_local=write_local)

    eng = fgd.Engine(M, P, ld, dtype, device=0, mix1_state=state)
    try:
        eng.set_topology_dict("mix1", t1)
        eng.set_topology_dict("mix2", t2)
        if subset:
            eng.set_mix2_subset(subset)
        n1, n2 = eng.num_cd_rows_split()
        assert (n1, n2) == (ref_cd1.shape[0], ref_cd2.shape[0])
        # Mix1 half.
        g_tp, g_v = _dev_rows(torch, tp, dtype), torch.from_numpy(v).cuda()
        g_x = _dev_rows(torch, np.zeros_like(tp), dtype)
        cd1 = torch.full((n1, M), float("nan"), dtype=torch.float64, device="cuda")
        eng.mix1(g_tp, g_x, g_v if state else None, cd1)
        torch.cuda.synchronize()
        got_x, got_vm = _host_rows(torch, g_x, dtype), g_v.cpu().numpy()
        scale = float(np.abs(tensors.bf16_bits_to_f32(tp) if dtype == "bf16" else tp).max())
        pa.compare_outputs(dtype, got_x, ref_x, got_vm, ref_vm if state else v, P, scale)
        assert np.array_equal(_host_rows(torch, g_tp, dtype), tp)  # theta_prev is only read
        pa.compare_cd(cd1.cpu().numpy(), ref_cd1, pa.cd_floor(P, scale))
        if ld > P:
            assert np.array_equal(got_x[:, P:], np.zeros_like(tp)[:, P:])
        # Blocking half from the oracle's stored x.
        g_x = _dev_rows(torch, ref_x, dtype)
        g_tp, g_tl = _dev_rows(torch, tp, dtype), _dev_rows(torch, tl, dtype)
        g_v = torch.from_numpy(np.ascontiguousarray(v_in)).cuda()
        cd2 = torch.full((n2, M), float("nan"), dtype=torch.float64, device="cuda")
        eng.outer_step_blocking(g_x, g_tp, g_tl, g_v, cd2, write_local=write_local)
        torch.cuda.synchronize()
        got_t, got_tl, got_v = _host_rows(torch, g_tp, dtype), _host_rows(torch, g_tl, dtype), g_v.cpu().numpy()
        pa.compare_outputs(dtype, got_t, ref_t, got_v, ref_v, P, scale)
        pa.compare_step_cd(cd2.cpu().numpy(), ref_cd2, ref_t, dtype, P, scale)
        if write_local:
            assert np.array_equal(got_tl[:, :P], got_t[:, :P])
        else:
            assert np.array_equal(got_tl, tl)
    finally:
        eng.close()


def test_split_round_on_two_streams(env):
    """A round as Algorithm 1 runs it: Mix1 on a side stream, a stand-in inner
    loop (matrix products) on the main stream, then the blocking half after
    waiting for Mix1; the result equals the oracle's two halves (float32
    storage: the engine's own x then differs from the oracle's by float32
    rounding only)."""
    fgd, torch = env
    M, P, dtype = 8, 200_003, "f32"
    ld = pa.aligned_ld(P)
    tp, tl, v = tensors.numpy_inputs(M, P, ld=ld, dtype=dtype, mom_std=1e-3, seed=61)
    t1, t2 = pa.topo(G, M, 1), pa.topo(RING_MH, M, 1, 3)
    ref_x, _, _ = oracle.mix1_split(tp, oracle.Mix.from_topology(t1), P=P)
    ref_t, ref_tl, ref_v, ref_cd2 = oracle.outer_blocking(ref_x, tp, tl, v, oracle.Mix.from_topology(t2), P=P,
                                                          write_local=True)
    eng = fgd.Engine(M, P, ld, dtype, device=0)
    try:
        eng.set_topology_dict("mix1", t1)
        eng.set_topology_dict("mix2", t2)
        g_tp, g_tl, g_v = _dev_rows(torch, tp, dtype), _dev_rows(torch, tl, dtype), torch.from_numpy(v).cuda()
        g_x = torch.empty_like(g_tp)
        side = torch.cuda.Stream()
        main = torch.cuda.current_stream()
        side.wait_stream(main)
        with torch.cuda.stream(side):
            eng.mix1(g_tp, g_x, None, None, side)
            done = torch.cuda.Event()
            done.record(side)
        a = torch.randn(2048, 2048, device="cuda", dtype=torch.float32)
        for _ in range(8):
            a = torch.tanh(a @ a) * 0.5
        main.wait_event(done)
        cd2 = torch.zeros((eng.num_cd_rows_split()[1], M), dtype=torch.float64, device="cuda")
        eng.outer_step_blocking(g_x, g_tp, g_tl, g_v, cd2, write_local=True, stream=main)
        torch.cuda.synchronize()
        scale = float(np.abs(tp).max())
        got_x = _host_rows(torch, g_x, dtype)
        pa.compare_outputs(dtype, got_x, ref_x, v, v, P, scale)
        got_t = _host_rows(torch, g_tp, dtype)
        pa.compare_outputs(dtype, got_t, ref_t, g_v.cpu().numpy(), ref_v, P, scale)
        assert np.array_equal(_host_rows(torch, g_tl, dtype)[:, :P], got_t[:, :P])
    finally:
        eng.close()


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_mix1_result_independent_of_block_count(env, dtype):
    """The Mix1 half takes chunks from a counter; x, the mixed momentum and
    the consensus rows are bit-identical for any number of blocks."""
    fgd, torch = env
    M, P = 8, 300_001
    ld = pa.aligned_ld(P)
    tp, _, v = tensors.numpy_inputs(M, P, ld=ld, dtype=dtype, mom_std=1e-3, seed=67)
    t1 = pa.topo(RING_MH, M, 2, 5)
    eng = fgd.Engine(M, P, ld, dtype, device=0, mix1_state=True)
    try:
        eng.set_topology_dict("mix1", t1)
        eng.set_topology("mix2", "identity")
        outs = []
        for nb in (0, 1, 7, 100, 5000):
            g_tp, g_v = _dev_rows(torch, tp, dtype), torch.from_numpy(v).cuda()
            g_x = torch.zeros_like(g_tp)
            cd = torch.zeros((eng.num_cd_rows_split()[0], M), dtype=torch.float64, device="cuda")
            eng.mix1(g_tp, g_x, g_v, cd, num_blocks=nb)
            torch.cuda.synchronize()
            outs.append((_host_rows(torch, g_x, dtype), g_v.cpu().numpy(), cd.cpu().numpy()))
        for o in outs[1:]:
            for a, b in zip(outs[0], o):
                assert np.array_equal(a, b)
    finally:
        eng.close()


def test_split_rejections(env):
    fgd, torch = env
    M, P = 4, 1024
    eng = fgd.Engine(M, P, P, "f32", device=0, mix1_state=True)
    try:
        eng.set_topology("mix1", "global")
        eng.set_topology("mix2", "global")
        a = torch.zeros((M, P), device="cuda")
        b, v = torch.zeros_like(a), torch.zeros_like(a)
        with pytest.raises(fgd.FgdError) as e:   # the state is mixed: momentum is required
            fgd.fgd_mix1(eng.handle, a, b, None)
        assert e.value.status == fgd.FGD_ERR_INVALID_ARG
        with pytest.raises(fgd.FgdError) as e:   # x aliases theta_prev
            fgd.fgd_mix1(eng.handle, a, a, v)
        assert e.value.status == fgd.FGD_ERR_INVALID_ARG
        with pytest.raises(fgd.FgdError) as e:   # negative block count
            fgd.fgd_mix1(eng.handle, a, b, v, None, -1)
        assert e.value.status == fgd.FGD_ERR_INVALID_ARG
        with pytest.raises(fgd.FgdError) as e:   # x aliases theta_local
            fgd.fgd_outer_step_blocking(eng.handle, b, a, b, v)
        assert e.value.status == fgd.FGD_ERR_INVALID_ARG
        eng.set_mix2_subset([(0, 10)])
        with pytest.raises(fgd.FgdError) as e:   # subset with a global Mix2
            fgd.fgd_outer_step_blocking(eng.handle, torch.zeros_like(a), a, b, v)
        assert e.value.status == fgd.FGD_ERR_UNSUPPORTED
    finally:
        eng.close()


def test_topology_ring_wraps_across_streams(env):
    """Twelve rounds on one engine that alternate the fused step and the split
    halves on two streams, with new edge masks every round: each round
    re-uploads the tables (a new mask, or a different stream), so the eight
    topology slots wrap several times while earlier launches may still be in
    flight.  Before each round the engine's arrays are loaded with the
    oracle's state (no engine output reaches the oracle); every round is
    checked."""
    fgd, torch = env
    M, P, dtype = 8, 20_011, "f32"
    ld = pa.aligned_ld(P)
    tp, tl, v = tensors.numpy_inputs(M, P, ld=ld, dtype=dtype, mom_std=1e-3, seed=73)
    t1 = pa.topo(G, M, 1)
    m1 = oracle.Mix.from_topology(t1)
    eng = fgd.Engine(M, P, ld, dtype, device=0)
    side = torch.cuda.Stream()
    main = torch.cuda.current_stream()
    try:
        eng.set_topology_dict("mix1", t1)
        g_tp, g_tl, g_v = (torch.from_numpy(a).cuda() for a in (tp, tl, v))
        g_x = torch.empty_like(g_tp)
        cur_t, cur_v = tp, v
        scale = float(np.abs(tp).max())
        for r in range(12):
            t2 = pa.topo(RING_MH, M, 1, seed=0, step=r)
            m2 = oracle.Mix.from_topology(t2)
            eng.set_topology_dict("mix2", t2)
            g_tp.copy_(torch.from_numpy(cur_t))
            g_v.copy_(torch.from_numpy(cur_v))
            if r % 2 == 0:
                ref_t, ref_v, _ = oracle.outer_step(cur_t, tl, cur_v, m1, m2, P=P)
                eng.outer_step(g_tp, g_tl, g_v, None, main)
            else:
                ref_x, _, _ = oracle.mix1_split(cur_t, m1, P=P)
                ref_t, _, ref_v, _ = oracle.outer_blocking(ref_x, cur_t, tl, cur_v, m2, P=P)
                side.wait_stream(main)
                with torch.cuda.stream(side):
                    eng.mix1(g_tp, g_x, None, None, side)
                    done = torch.cuda.Event()
                    done.record(side)
                main.wait_event(done)
                eng.outer_step_blocking(g_x, g_tp, g_tl, g_v, None, stream=main)
            torch.cuda.synchronize()
            pa.compare_outputs(dtype, g_tp.cpu().numpy(), ref_t, g_v.cpu().numpy(), ref_v, P, scale)
            cur_t, cur_v = ref_t, ref_v
    finally:
        eng.close()
