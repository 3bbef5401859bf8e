"""GPU parity on the edge cases the oracle defines: non-finite values, links
dropped for a round, and subnormal float32 values, through the C ABI.

  masked links   A link dropped for a round contributes nothing to it
                 (Sec. 3 mixing over the live graph): an infinity or NaN in
                 the dropped neighbour must not reach the worker, in the fused
                 step and in the blocking half of split execution.  A kernel
                 that kept dropped entries with weight 0 would pass every
                 finite case (0 * x = 0) and fail these (0 * inf = NaN).
  non-finite     NaN and infinities in theta_prev, theta_local or the
                 momentum propagate exactly where the oracle's do: the same
                 elements of theta' and v' are NaN or infinite (with the same
                 sign), and so are the same consensus entries.
  row padding    elements in [P, ld) of every row are read with the lane
                 vectors that straddle P but never enter the step, its sums
                 or its consensus, and are never written.
  subnormal      float32 subnormals are kept, not flushed: with g0 = 0 the
                 momentum update v' = mu v is one rounding of an exact product
                 on both sides, so v' matches the oracle bit for bit; with
                 lr = 1, mu = 1/2 and multiples of four subnormal units every
                 operation is exact and theta' matches bit for bit too.
"""

import numpy as np
import pytest

import oracle
from synth import graphs, tensors
from tests import _parity as pa

pytestmark = pytest.mark.gpu

RING_MH = ("ring", "metropolis", 0.1)
REG4 = ("regular", "metropolis", 4)
G, ID = ("global",), ("identity",)


@pytest.fixture(scope="module")
def env():
    import torch

    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    import paper_2606_22768_amd as fgd

    return fgd, torch


def _finite_scale(a, dtype):
    v = tensors.bf16_bits_to_f32(a) if dtype == "bf16" else np.asarray(a, np.float32)
    v = np.abs(v[np.isfinite(v)])
    return float(v.max()) if v.size else 0.0


def _set(a, dtype, m, p, value):
    """a[m, p] = value (float), in the storage of a."""
    if dtype == "bf16" and a.dtype == np.uint16:
        a[m, p] = tensors.f32_to_bf16_bits(np.array([value], np.float32))[0]
    else:
        a[m, p] = value


def _dropped_ring(M, rounds, dropped, reweight="metropolis"):
    """Ring topology whose links in `dropped` (undirected pairs) are masked in
    every round; the rest are live."""
    rp, ci, w = graphs.ring_weights(M)
    live = [e for e in graphs.undirected_edges(rp, ci) if tuple(sorted(e)) not in dropped]
    masks = graphs.masks_from_live_edges(rp, ci, [live] * rounds)
    return dict(kind="csr", row_ptr=rp, col_idx=ci, weights=w if reweight == "self" else None, rounds=rounds,
                masks=masks, reweight=reweight)


def _fused(env, M, P, dtype, t1, t2, tp, tl, v, lr=0.7, mu=0.9):
    fgd, torch = env
    ld = tp.shape[1]
    ref_t, ref_v, ref_cd = oracle.outer_step(tp, tl, v, oracle.Mix.from_topology(t1), oracle.Mix.from_topology(t2),
                                             lr=lr, mu=mu, P=P, dtype=dtype)
    got_t, got_v, got_cd = pa.run_engine(fgd, torch, M, P, ld, dtype, t1, t2, tp, tl, v, True, lr, mu)
    scale = _finite_scale(tp[:, :P], dtype)
    pa.compare_outputs(dtype, got_t, ref_t, got_v, ref_v, P, scale)
    pa.compare_step_cd(got_cd, ref_cd, ref_t, dtype, P, scale)
    return (got_t, got_v, got_cd), (ref_t, ref_v, ref_cd)


def _blocking(env, M, P, dtype, t1, t2, tp, tl, v, write_local=True):
    """Blocking half fed the oracle's stored Mix1 output."""
    fgd, torch = env
    ld = tp.shape[1]
    m1, m2 = oracle.Mix.from_topology(t1), oracle.Mix.from_topology(t2)
    ref_x, _, _ = oracle.mix1_split(tp, m1, mom=v, P=P)
    ref_t, ref_tl, ref_v, ref_cd = oracle.outer_blocking(ref_x, tp, tl, v, m2, P=P, write_local=write_local)

    def dev(a):
        t = torch.from_numpy(np.ascontiguousarray(a.view(np.int16) if dtype == "bf16" else a)).cuda()
        return t.view(torch.bfloat16) if dtype == "bf16" else t

    def host(t):
        return t.view(torch.int16).cpu().numpy().view(np.uint16) if dtype == "bf16" else t.cpu().numpy()

    eng = fgd.Engine(M, P, ld, dtype, device=0)
    try:
        eng.set_topology_dict("mix1", t1)
        eng.set_topology_dict("mix2", t2)
        g_x, g_tp, g_tl, g_v = dev(ref_x), dev(tp), dev(tl), torch.from_numpy(np.ascontiguousarray(v)).cuda()
        cd = torch.full((eng.num_cd_rows_split()[1], M), 0.5, dtype=torch.float64, device="cuda")
        eng.outer_step_blocking(g_x, g_tp, g_tl, g_v, cd, write_local=write_local)
        torch.cuda.synchronize()
        got_t, got_tl, got_v, got_cd = host(g_tp), host(g_tl), g_v.cpu().numpy(), cd.cpu().numpy()
    finally:
        eng.close()
    scale = _finite_scale(tp[:, :P], dtype)
    pa.compare_outputs(dtype, got_t, ref_t, got_v, ref_v, P, scale)
    pa.compare_step_cd(got_cd, ref_cd, ref_t, dtype, P, scale)
    if write_local:
        pa.compare_outputs(dtype, got_tl, ref_tl, got_v, ref_v, P, scale)
    return got_t, got_v


# ------------------------------------------------------------ masked links

BAD = [np.inf, -np.inf, np.nan]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("reweight", ["metropolis", "self"])
@pytest.mark.parametrize("rounds", [1, 2])
def test_dropped_link_does_not_leak_non_finite_values(env, dtype, reweight, rounds):
    """Link (2, 3) of a ring of 8 is dropped in every Mix2 round; worker 3's
    local parameters hold +inf, -inf and NaN at three indices, so its outer
    gradient does too.  Worker 2 pulls only from 1 and itself: its theta' and
    v' stay finite there and match the oracle; worker 3 and the workers the
    values reach through live links are non-finite exactly as in the oracle."""
    M, P = 8, 2 * 1024 + 37
    ld = pa.aligned_ld(P)
    print(f"[edge] dropped link, fused, {dtype} {reweight} rounds={rounds}", flush=True)
    tp, tl, v = tensors.numpy_inputs(M, P, ld=ld, dtype=dtype, seed=3)
    idx = [5, 1031, P - 1]
    for p, bad in zip(idx, BAD):
        _set(tl, dtype, 3, p, bad)
    t2 = _dropped_ring(M, rounds, {(2, 3)}, reweight)
    (got_t, got_v, got_cd), _ = _fused(env, M, P, dtype, pa.topo(G, M, 1), t2, tp, tl, v)
    vals = tensors.bf16_bits_to_f32(got_t) if dtype == "bf16" else got_t
    assert np.isfinite(vals[2, idx]).all() and np.isfinite(got_v[2, idx]).all()
    assert not np.isfinite(got_v[3, idx]).any()


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_dropped_link_in_both_mixes(env, dtype):
    """LocalM1M2 with link (2, 3) dropped in Mix1 and Mix2: a NaN in worker
    3's previous parameters reaches neither worker 2's mixed parameters nor
    its mixed gradient."""
    M, P = 8, 1500
    ld = pa.aligned_ld(P)
    print(f"[edge] dropped link in both mixes, {dtype}", flush=True)
    tp, tl, v = tensors.numpy_inputs(M, P, ld=ld, dtype=dtype, seed=4)
    _set(tp, dtype, 3, 700, np.nan)
    _set(tp, dtype, 3, 701, np.inf)
    t = _dropped_ring(M, 1, {(2, 3)})
    (got_t, got_v, _), _ = _fused(env, M, P, dtype, t, t, tp, tl, v)
    vals = tensors.bf16_bits_to_f32(got_t) if dtype == "bf16" else got_t
    assert np.isfinite(vals[2, 700:702]).all() and np.isfinite(got_v[2, 700:702]).all()


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_dropped_link_in_the_blocking_half(env, dtype):
    """Split execution: the blocking half's Mix2 drops link (2, 3) as well."""
    M, P = 8, 3079
    ld = pa.aligned_ld(P)
    print(f"[edge] dropped link, blocking half, {dtype}", flush=True)
    tp, tl, v = tensors.numpy_inputs(M, P, ld=ld, dtype=dtype, seed=5)
    for p, bad in zip([0, 100, P - 2], BAD):
        _set(tl, dtype, 3, p, bad)
    t1 = _dropped_ring(M, 1, {(2, 3)})
    t2 = _dropped_ring(M, 2, {(2, 3)}, "self")
    got_t, got_v = _blocking(env, M, P, dtype, t1, t2, tp, tl, v)
    vals = tensors.bf16_bits_to_f32(got_t) if dtype == "bf16" else got_t
    assert np.isfinite(vals[2, [0, 100, P - 2]]).all() and np.isfinite(got_v[2, [0, 100, P - 2]]).all()


# ------------------------------------------------------- non-finite inputs

# (M, P, dtype, mix1, K1, mix2, K2)
PROPAGATION = [
    (8, 4 * 1024 + 3, "bf16", G, 1, RING_MH, 1),    # GlobalM1LocalM2 (the bf16 workload's kinds)
    (8, 4 * 1024 + 3, "f32", ID, 0, G, 1),          # DiLoCo
    (16, 3 * 1024 + 9, "f32", G, 1, ("exp", "given"), 2),
    (64, 777, "f32", REG4, 1, REG4, 3),             # LocalM1M2 at 64 workers (the consensus-every-round workload)
    (64, 777, "bf16", G, 1, REG4, 2),
    (5, 1001, "f32", ("er_mh", 0.6, 0.2), 2, ("ring_self", 0.3), 1),  # run-time worker count
    (32, 513, "f32", REG4, 2, G, 1),
]


@pytest.mark.parametrize("case", PROPAGATION, ids=lambda c: f"M{c[0]}-P{c[1]}-{c[2]}-{c[3][0]}{c[4]}-{c[5][0]}{c[6]}")
@pytest.mark.parametrize("where", ["theta_prev", "theta_local", "momentum", "all"])
def test_non_finite_values_propagate_like_the_oracle(env, case, where):
    """+inf, -inf and NaN at a few (worker, parameter) positions; every other
    column stays finite, so both the propagated values and the untouched
    ones are compared."""
    M, P, dtype, s1, k1, s2, k2 = case
    ld = pa.aligned_ld(P)
    print(f"[edge] non-finite in {where}: {case}", flush=True)
    tp, tl, v = tensors.numpy_inputs(M, P, ld=ld, dtype=dtype, seed=11)
    rng = np.random.default_rng(17)
    targets = {"theta_prev": [tp], "theta_local": [tl], "momentum": [v], "all": [tp, tl, v]}[where]
    for a in targets:
        for bad in BAD:
            m, p = int(rng.integers(0, M)), int(rng.integers(0, P))
            _set(a, dtype, m, p, bad)
    t1, t2 = pa.topo(s1, M, k1, 2), pa.topo(s2, M, k2, 9)
    _fused(env, M, P, dtype, t1, t2, tp, tl, v)


def test_opposite_infinities_in_one_column(env):
    """+inf and -inf at the same parameter of two workers: the global mean
    there is NaN, so every worker's theta' there is NaN, and every S_m of the
    rows whose mean includes that column is NaN (the global-mean output row
    too: mean - mean is NaN for a non-finite mean)."""
    M, P = 8, 1100
    ld = pa.aligned_ld(P)
    print("[edge] opposite infinities", flush=True)
    tp, tl, v = tensors.numpy_inputs(M, P, ld=ld, dtype="f32", seed=12)
    tp[1, 40], tp[6, 40] = np.inf, -np.inf
    (got_t, _, got_cd), _ = _fused(env, M, P, "f32", pa.topo(G, M, 1), pa.topo(RING_MH, M, 1, 3), tp, tl, v)
    assert np.isnan(got_t[:, 40]).all()
    assert np.isnan(got_cd[-1]).all()


# --------------------------------------------------------------- subnormals

def _subnormals(rng, shape, multiple=1):
    """float32 subnormals k * 2^-149, k a random multiple of `multiple` in
    [multiple, 2^23), random sign."""
    k = rng.integers(1, (1 << 23) // multiple, size=shape) * multiple
    s = np.where(rng.integers(0, 2, size=shape) == 1, np.uint32(0x80000000), np.uint32(0))
    return (k.astype(np.uint32) | s).view(np.float32)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("mix1", [ID, G])
def test_subnormal_momentum_is_kept(env, dtype, mix1):
    """g0 = 0 (theta_local = theta_prev; every Mix2 round of zeros is 0) and
    subnormal momentum: v' = mu v is one rounding of an exact product in the
    kernel (an FMA with addend 0) and in the oracle (an exact double product
    rounded once to float32), so v' must match bit for bit; a flush of
    subnormals to zero would give 0.  The global mean runs over equal rows
    (every worker holds the same theta_prev), which it reproduces exactly."""
    M, P = 8, 2 * 1024 + 5
    ld = pa.aligned_ld(P)
    print(f"[edge] subnormal momentum {dtype} mix1={mix1[0]}", flush=True)
    tp, _, _ = tensors.numpy_inputs(M, P, ld=ld, dtype=dtype, seed=21)
    tp[:] = tp[0]
    tl = tp.copy()
    v = np.zeros((M, ld), np.float32)
    v[:, :P] = _subnormals(np.random.default_rng(22), (M, P))
    (got_t, got_v, _), (ref_t, ref_v, _) = _fused(env, M, P, dtype, pa.topo(mix1, M, 1), pa.topo(RING_MH, M, 1, 5),
                                                  tp, tl, v)
    assert np.array_equal(got_v[:, :P].view(np.uint32), ref_v[:, :P].view(np.uint32))
    assert (np.abs(got_v[:, :P]) < np.float32(2.0 ** -126)).mean() > 0.9  # mostly still subnormal
    assert np.array_equal(got_t[:, :P], ref_t[:, :P])  # theta' = x: the update is far below half an ulp


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_subnormal_parameters_exact_step(env, dtype):
    """Subnormal parameters and momentum with lr = 1, mu = 1/2: theta_prev a
    subnormal (float32: k 2^-149; bf16: k 2^-133), v = 4 j units, g0 = 0.
    Then v' = v / 2, step = v' / 2 and theta' = x - step are exact in both
    implementations, so theta' and v' match bit for bit."""
    M, P = 8, 1024 + 77
    ld = pa.aligned_ld(P)
    print(f"[edge] subnormal parameters {dtype}", flush=True)
    rng = np.random.default_rng(31)
    if dtype == "f32":
        tp = np.zeros((M, ld), np.float32)
        tp[:, :P] = _subnormals(rng, (M, P))
        v = np.zeros((M, ld), np.float32)
        v[:, :P] = _subnormals(rng, (M, P), multiple=4)
    else:
        k = rng.integers(1, 128, size=(M, P)).astype(np.uint16)  # bf16 subnormals: k * 2^-133
        tp = np.zeros((M, ld), np.uint16)
        tp[:, :P] = k | np.where(rng.integers(0, 2, size=(M, P)) == 1, np.uint16(0x8000), np.uint16(0))
        j = rng.integers(1, 32, size=(M, P)).astype(np.float64)
        v = np.zeros((M, ld), np.float32)
        v[:, :P] = (4 * j * 2.0 ** -133 * np.where(rng.integers(0, 2, size=(M, P)) == 1, -1, 1)).astype(np.float32)
    tl = tp.copy()
    (got_t, got_v, _), (ref_t, ref_v, _) = _fused(env, M, P, dtype, pa.topo(ID, M, 0), pa.topo(RING_MH, M, 1, 6),
                                                  tp, tl, v, lr=1.0, mu=0.5)
    assert np.array_equal(got_v[:, :P].view(np.uint32), ref_v[:, :P].view(np.uint32))
    if dtype == "f32":
        assert np.array_equal(got_t[:, :P].view(np.uint32), ref_t[:, :P].view(np.uint32))
    else:
        assert np.array_equal(got_t[:, :P], ref_t[:, :P])


PAD_CASES = [
    # (M, P, dtype, mix1, k1, mix2, k2): the lane-per-parameter kernel and the worker-group kernel
    (8, 3 * 1024 + 5, "bf16", G, 1, RING_MH, 1),
    (8, 777, "f32", G, 1, RING_MH, 1),
    (64, 2 * 256 + 3, "f32", REG4, 1, REG4, 3),
]


@pytest.mark.parametrize("case", PAD_CASES, ids=lambda c: f"M{c[0]}-P{c[1]}-{c[2]}")
def test_row_padding_is_never_used(env, case):
    """NaN, infinities and huge values in [P, ld) of theta_prev, theta_local
    and the momentum give bit-identical outputs and consensus rows to zero
    padding, and stay as they were."""
    fgd, torch = env
    M, P, dtype, s1, k1, s2, k2 = case
    ld = pa.aligned_ld(P) + 8  # a ragged last lane vector and whole vectors of padding
    tp, tl, v = tensors.numpy_inputs(M, P, ld=ld, dtype=dtype, seed=5)
    for a in (tp, tl, v):
        a[:, P:] = 0
    t1, t2 = pa.topo(s1, M, k1, 3), pa.topo(s2, M, k2, 4)
    ref = pa.run_engine(fgd, torch, M, P, ld, dtype, t1, t2, tp.copy(), tl.copy(), v.copy())
    junk = np.array([np.nan, np.inf, -np.inf, 3e38, -3e38], np.float32)
    for a in (tp, tl, v):
        fill = np.resize(junk, a[:, P:].shape)
        a[:, P:] = tensors.f32_to_bf16_bits(fill) if a.dtype == np.uint16 else fill
    got = pa.run_engine(fgd, torch, M, P, ld, dtype, t1, t2, tp.copy(), tl.copy(), v.copy())
    for r, g, what in zip(ref, got, ("theta'", "v'", "consensus rows")):
        r, g = np.asarray(r), np.asarray(g)
        if what == "consensus rows":
            assert np.array_equal(r, g), what
        else:
            assert np.array_equal(r[:, :P], g[:, :P]), what
    # bit patterns: NaN padding compares unequal to itself as floats
    bits = lambda a: np.ascontiguousarray(a).view(np.uint16 if a.dtype == np.uint16 else np.uint32)
    assert np.array_equal(bits(np.asarray(got[0])[:, P:]), bits(tp[:, P:]))
    assert np.array_equal(bits(np.asarray(got[1])[:, P:]), bits(v[:, P:]))
