"""Full-size parity at the benchmark's launch configuration, for the four
large workloads (8x150M f32, 16x500M f32, 8x1.1e9 bf16, 64x124M f32).

Outputs are checked element by element against the oracle on sampled
parameter columns (every column is independent given W, so the oracle run on
the gathered columns is exact parity for them): the first and last columns
(ragged end of the tiles) and seeded random ones.  The consensus rows, which
the oracle cannot recompute at this size, are checked through properties that
hold at any size:
  - x^0 row = standalone consensus kernel on theta_prev before the step;
  - g^0 row = standalone consensus kernel on theta_prev - theta_local
    (formed by torch in float32, the same single rounding the kernel does);
  - theta' row = standalone consensus kernel on the stored output;
  - a global-mean round leaves an exactly zero row;
  - each CSR round contracts: S(W u) <= sigma_2(W)^2 S(u), sigma_2 from the
    round's effective weights (Sec. 3 contraction factor); with a Mix2 subset
    only S(round) <= S(input) holds, since the rest passes through.
The step variants (Mix1 over the momentum, Mix2 on a 43% subset) run on the
8 x 1.1e9 bf16 inputs.
"""

import gc

import numpy as np
import pytest
import scipy.sparse

import oracle
from synth import configs, tensors
from tests import _parity as pa

pytestmark = pytest.mark.gpu

WORKLOADS = ["m8_p150m_f32", "m16_p500m_f32", "m8_p1100m_bf16", "m64_p124m_f32", "m8_p1100m_bf16_m1s_subset43"]


@pytest.fixture(scope="module")
def env():
    import torch

    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    import paper_2606_22768_amd as fgd

    return fgd, torch


def _sample_columns(P, seed, n_edge=2048, n_random=8192):
    rng = np.random.default_rng(seed)
    cols = set(range(min(n_edge, P)))
    cols |= set(range(max(0, P - n_edge), P))
    cols |= set(rng.integers(0, P, n_random).tolist())
    return np.array(sorted(cols), dtype=np.int64)


def _segments_in_sample(cols, segs):
    """The subset as segments of the gathered column index space."""
    if segs is None:
        return None
    inside = np.zeros(len(cols), dtype=bool)
    for b, e in segs.tolist():
        inside |= (cols >= b) & (cols < e)
    out, j = [], 0
    while j < len(cols):
        if inside[j]:
            k = j
            while k < len(cols) and inside[k]:
                k += 1
            out.append((j, k))
            j = k
        else:
            j += 1
    return out


def _host(t, dtype):
    import torch

    t = t.contiguous()
    return t.view(torch.int16).cpu().numpy().view(np.uint16) if dtype == "bf16" else t.cpu().numpy()


def _sigma2(row_ptr, col_idx, w):
    M = len(row_ptr) - 1
    W = scipy.sparse.csr_matrix((np.asarray(w, np.float64), col_idx, row_ptr), shape=(M, M)).toarray()
    s = np.linalg.svd(W, compute_uv=False)
    return sorted(s)[-2]


@pytest.mark.parametrize("workload", WORKLOADS)
def test_fullsize_step(env, workload):
    fgd, torch = env
    w = configs.WORKLOADS[workload]
    M, P, dtype = w["M"], w["P"], w["dtype"]
    ld = pa.aligned_ld(P)
    state = bool(w.get("mix1_state"))
    eng = fgd.Engine(M, P, ld, dtype, configs.OUTER_LR, configs.MOMENTUM, device=0, mix1_state=state)
    # The arrays are placed as bench.py places them (one spread buffer).
    st = eng.alloc_state(spread=True)
    print(f"[fullsize] {workload}: generating inputs", flush=True)
    tp, tl, v = tensors.torch_inputs(M, P, ld=ld, dtype=dtype, prev_std=w["prev_std"], drift_std=w["drift_std"],
                                     mom_std=w["mom_std"], seed=w["seed"], device="cuda",
                                     out=(st["theta_prev"], st["theta_local"], st["momentum"]))
    cols = _sample_columns(P, w["seed"])
    icol = torch.from_numpy(cols).cuda()
    s_tp, s_tl, s_v = (_host(t.index_select(1, icol), d) for t, d in ((tp, dtype), (tl, dtype), (v, "f32")))

    t1 = configs.topology(w["mix1"], M, w["k1"], w["seed"])
    t2 = configs.topology(w["mix2"], M, w["k2"], w["seed"], step=0)
    segs = configs.subset_segments(w)
    eng.set_topology_dict("mix1", t1)
    eng.set_topology_dict("mix2", t2)
    if segs is not None:
        eng.set_mix2_subset(segs)
    n_rows = eng.num_cd_rows()

    # Standalone consensus of the inputs, by a different kernel.
    cd_x0 = torch.zeros(M, dtype=torch.float64, device="cuda")
    eng.consensus_distance(tp, cd_x0)
    g0 = tp[:, :P].float() - tl[:, :P].float()
    g0_full = torch.zeros((M, ld), dtype=torch.float32, device="cuda")
    g0_full[:, :P] = g0
    del g0
    cd_g0 = torch.zeros(M, dtype=torch.float64, device="cuda")
    eng.consensus_distance(g0_full, cd_g0, dtype="f32")
    torch.cuda.synchronize()
    del g0_full
    gc.collect()
    torch.cuda.empty_cache()

    print(f"[fullsize] {workload}: step", flush=True)
    cd = torch.full((n_rows, M), float("nan"), dtype=torch.float64, device="cuda")
    eng.outer_step(tp, tl, v, cd)
    cd_out = torch.zeros(M, dtype=torch.float64, device="cuda")
    eng.consensus_distance(tp, cd_out)
    torch.cuda.synchronize()
    got_t = _host(tp.index_select(1, icol), dtype)
    got_v = _host(v.index_select(1, icol), "f32")
    cd = cd.cpu().numpy()

    # Element-by-element parity on the sampled columns.
    s_segs = _segments_in_sample(cols, segs)
    m2 = oracle.Mix.from_topology(t2) if (s_segs is None or s_segs) else oracle.Mix("identity")
    ref_t, ref_v, _ = oracle.outer_step(s_tp, s_tl, s_v, oracle.Mix.from_topology(t1), m2,
                                        lr=configs.OUTER_LR, mu=configs.MOMENTUM, dtype=dtype, mix1_state=state,
                                        subset=s_segs if s_segs else None)
    scale = float(np.abs(tensors.bf16_bits_to_f32(s_tp) if dtype == "bf16" else s_tp).max())
    pa.compare_outputs(dtype, got_t, ref_t, got_v, ref_v, len(cols), scale)

    # Consensus rows.
    k2 = 1 if t2["kind"] == "global" else t2["rounds"]
    k1 = 1 if t1["kind"] == "global" else t1["rounds"]
    assert n_rows == k2 + k1 + 3
    np.testing.assert_allclose(cd[0], cd_g0.cpu().numpy(), rtol=1e-9)
    np.testing.assert_allclose(cd[k2 + 1], cd_x0.cpu().numpy(), rtol=1e-9)
    np.testing.assert_allclose(cd[-1], cd_out.cpu().numpy(), rtol=1e-9)
    for t, first in ((t2, 0), (t1, k2 + 1)):
        K = 1 if t["kind"] == "global" else t["rounds"]
        for k in range(K):
            before, after = cd[first + k].sum(), cd[first + k + 1].sum()
            if t["kind"] == "global":
                assert np.all(cd[first + k + 1] == 0.0)
                continue
            which = "mix2" if t is t2 else "mix1"
            s2 = _sigma2(t["row_ptr"], t["col_idx"], eng.effective_weights(which, k))
            if which == "mix2" and segs is not None:
                s2 = 1.0
            assert after <= s2 ** 2 * before * (1 + 1e-5), (workload, which, k, after / before, s2 ** 2)
    print(f"[fullsize] {workload}: ok, consensus rows {np.round(cd.mean(axis=1), 6).tolist()}", flush=True)
    eng.close()
    del tp, tl, v, st, cd_x0, cd_g0, cd_out
    gc.collect()
    torch.cuda.empty_cache()


def test_fullsize_split_round(env):
    """Split execution at the size and launch configuration of `bench.py
    --mode split` (8 x 1.1e9 bf16, one spread buffer with x, Mix1 half on 128
    blocks, blocking half with the write-back into theta_local), element by
    element on sampled columns.  The blocking half runs from the oracle's x at
    the sampled columns (written into the engine's x there), so no engine
    output feeds the oracle."""
    fgd, torch = env
    name = "m8_p1100m_bf16"
    w = configs.WORKLOADS[name]
    M, P, dtype = w["M"], w["P"], w["dtype"]
    ld = pa.aligned_ld(P)
    eng = fgd.Engine(M, P, ld, dtype, configs.OUTER_LR, configs.MOMENTUM, device=0)
    st = eng.alloc_state(spread=True, with_x=True)
    print(f"[fullsize] split {name}: generating inputs", flush=True)
    tp, tl, v = tensors.torch_inputs(M, P, ld=ld, dtype=dtype, prev_std=w["prev_std"], drift_std=w["drift_std"],
                                     mom_std=w["mom_std"], seed=w["seed"], device="cuda",
                                     out=(st["theta_prev"], st["theta_local"], st["momentum"]))
    x = st["x"]
    cols = _sample_columns(P, w["seed"] + 5)
    icol = torch.from_numpy(cols).cuda()
    s_tp, s_tl, s_v = (_host(t.index_select(1, icol), d) for t, d in ((tp, dtype), (tl, dtype), (v, "f32")))
    t1 = configs.topology(w["mix1"], M, w["k1"], w["seed"])
    t2 = configs.topology(w["mix2"], M, w["k2"], w["seed"], step=3)
    eng.set_topology_dict("mix1", t1)
    eng.set_topology_dict("mix2", t2)
    n1, n2 = eng.num_cd_rows_split()
    cd_x0 = torch.zeros(M, dtype=torch.float64, device="cuda")
    eng.consensus_distance(tp, cd_x0)

    print(f"[fullsize] split {name}: Mix1 half", flush=True)
    cd1 = torch.full((n1, M), float("nan"), dtype=torch.float64, device="cuda")
    eng.mix1(tp, x, None, cd1, num_blocks=128)
    torch.cuda.synchronize()
    got_x = _host(x.index_select(1, icol), dtype)
    ref_x, _, _ = oracle.mix1_split(s_tp, oracle.Mix.from_topology(t1), dtype=dtype)
    scale = float(np.abs(tensors.bf16_bits_to_f32(s_tp)).max())
    d = np.abs(pa.ordered_bf16(got_x) - pa.ordered_bf16(ref_x))
    assert d.max() <= 1, f"x differs by {d.max()} bf16 ulps"
    cd1 = cd1.cpu().numpy()
    np.testing.assert_allclose(cd1[0], cd_x0.cpu().numpy(), rtol=1e-9)   # x^0 row = theta_prev's consensus
    assert np.all(cd1[1] == 0.0)                                         # a global mean leaves no disagreement

    print(f"[fullsize] split {name}: blocking half", flush=True)
    xs = torch.from_numpy(ref_x.view(np.int16)).cuda().view(torch.bfloat16)
    x.index_copy_(1, icol, xs)
    cd2 = torch.full((n2, M), float("nan"), dtype=torch.float64, device="cuda")
    eng.outer_step_blocking(x, tp, tl, v, cd2, write_local=True)
    cd_out = torch.zeros(M, dtype=torch.float64, device="cuda")
    eng.consensus_distance(tp, cd_out)
    torch.cuda.synchronize()
    got_t, got_tl = _host(tp.index_select(1, icol), dtype), _host(tl.index_select(1, icol), dtype)
    got_v = _host(v.index_select(1, icol), "f32")
    ref_t, _, ref_v, _ = oracle.outer_blocking(ref_x, s_tp, s_tl, s_v, oracle.Mix.from_topology(t2),
                                               lr=configs.OUTER_LR, mu=configs.MOMENTUM, dtype=dtype,
                                               write_local=True)
    pa.compare_outputs(dtype, got_t, ref_t, got_v, ref_v, len(cols), scale)
    assert np.array_equal(got_tl, got_t)                                 # theta' written back as the next y_0
    cd2 = cd2.cpu().numpy()
    np.testing.assert_allclose(cd2[-1], cd_out.cpu().numpy(), rtol=1e-9)  # theta' row = standalone consensus
    s2 = _sigma2(t2["row_ptr"], t2["col_idx"], eng.effective_weights("mix2", 0))
    assert cd2[1].sum() <= s2 ** 2 * cd2[0].sum() * (1 + 1e-5)
    print(f"[fullsize] split {name}: ok", flush=True)
    eng.close()
    del tp, tl, v, x, st, cd_x0, cd_out
    gc.collect()
    torch.cuda.empty_cache()
