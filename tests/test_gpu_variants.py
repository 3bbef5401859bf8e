"""GPU parity of the step variants against the CPU oracle, element by element
and for every consensus row, through the C ABI:

  - plain momentum (Nesterov off);
  - Mix1 over the optimizer state (Appendix B, GlobalM1S / GlobalM1SLocalM2),
    on the specialised kernels and on the run-time-kind kernels;
  - Mix2 on a subset of parameter segments (Sec. 4.1 / Appendix C,
    GlobalM1LocalM2-subset), with segments aligned to tiles, inside a tile,
    a single element, at the ragged end, touching each other, and the
    combination with the state mix.
Sizes span several 256-lane tiles and end in a ragged tail.
"""

import numpy as np
import pytest

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

# (M, P, dtype, mix1, K1, mix2, K2)
PLAIN = [
    (1, 2051, "f32", ID, 0, ID, 0),
    (8, 3079, "bf16", G, 1, RING_MH, 1),
    (8, 3079, "f32", ID, 0, G, 1),
    (5, 2051, "f32", ("er_mh", 0.6, 0.2), 2, ("ring_self", 0.3), 1),
    (64, 775, "f32", REG4, 1, REG4, 3),
]


@pytest.mark.parametrize("case", PLAIN, ids=lambda c: f"M{c[0]}-{c[2]}-{c[3][0]}{c[4]}-{c[5][0]}{c[6]}")
def test_plain_momentum(env, case):
    fgd, torch = env
    M, P, dtype, s1, k1, s2, k2 = case
    print(f"[variants] plain momentum {case}", flush=True)
    pa.run_case(fgd, torch, M, P, dtype, s1, k1, s2, k2, seed=31, mom_std=1e-3, nesterov=False)


STATE = [
    (8, 3079, "bf16", G, 1, ID, 0),          # GlobalM1S (specialised)
    (8, 3079, "f32", G, 1, RING_MH, 1),      # GlobalM1SLocalM2 (specialised)
    (8, 3079, "bf16", G, 1, RING, 1),
    (16, 3079, "f32", G, 1, EXP, 2),
    (64, 775, "f32", REG4, 1, REG4, 3),      # CSR Mix1 on the state (run-time kinds)
    (8, 3079, "f32", ("matching",), 2, ("matching",), 1),
    (8, 3079, "f32", ID, 0, G, 1),           # identity Mix1: the state is unchanged
    (5, 2051, "bf16", G, 1, ("ring_self", 0.3), 2),  # M not a power of two
    (32, 900, "f32", ("er_mh", 0.2, 0.1), 2, G, 1),
    (1, 999, "f32", G, 1, ID, 0),
]


@pytest.mark.parametrize("case", STATE, ids=lambda c: f"M{c[0]}-{c[2]}-{c[3][0]}{c[4]}-{c[5][0]}{c[6]}")
@pytest.mark.parametrize("nesterov", [True, False], ids=["nesterov", "plain"])
def test_state_mix(env, case, nesterov):
    fgd, torch = env
    M, P, dtype, s1, k1, s2, k2 = case
    print(f"[variants] state mix {case} nesterov={nesterov}", flush=True)
    pa.run_case(fgd, torch, M, P, dtype, s1, k1, s2, k2, seed=37, mom_std=1e-3, nesterov=nesterov,
                mix1_state=True)


# Tiles hold 256 * V parameters: 1024 for V = 4 (M <= 16), 512 for V = 2
# (M = 32), 256 for V = 1 (M = 64).
SUBSETS = [
    [(0, 1024)],                                  # exactly the first tile
    [(37, 38)],                                   # one element
    [(1000, 3100), (5000, 5001), (9990, 10007)],  # straddling tiles, ragged end
    [(0, 5), (5, 1500), (1500, 1501)],            # touching segments
    [(0, 10007)],                                 # everything: equals the full Mix2
    [(4096, 8192)],                               # tile-aligned, middle
]


@pytest.mark.parametrize("segs", SUBSETS, ids=lambda s: f"{len(s)}seg-{s[0][0]}")
@pytest.mark.parametrize("case", [
    (8, "bf16", G, 1, RING_MH, 1, False),   # GlobalM1LocalM2-subset
    (8, "f32", G, 1, RING, 1, True),        # GlobalM1SLocalM2-subset
    (16, "f32", G, 1, EXP, 2, False),
    (64, "f32", REG4, 1, REG4, 3, False),
    (5, "bf16", ("er_mh", 0.6, 0.2), 1, ("ring_self", 0.3), 2, True),
], ids=lambda c: f"M{c[0]}-{c[1]}-{c[2][0]}{c[3]}-{c[4][0]}{c[5]}-state{int(c[6])}")
def test_subset(env, case, segs):
    fgd, torch = env
    M, dtype, s1, k1, s2, k2, state = case
    P = 10007
    print(f"[variants] subset {case} {segs}", flush=True)
    pa.run_case(fgd, torch, M, P, dtype, s1, k1, s2, k2, seed=41, mom_std=1e-3, mix1_state=state, subset=segs)


def _dense_segments(n, seed):
    """n ascending, disjoint half-open segments, one in each cell of 3
    parameters: lengths 1 to 3, some touching the next one."""
    rng = np.random.default_rng(seed)
    return [(3 * i + int(rng.integers(0, 2)), 3 * i + 3 - int(rng.integers(0, 2))) for i in range(n)]


@pytest.mark.parametrize("case", [
    (8, "bf16", G, 1, RING_MH, 1, False),   # about 340 segments in every 1024-parameter tile
    (8, "f32", G, 1, RING, 1, True),
    (64, "f32", REG4, 1, REG4, 3, False),   # about 85 segments in every 256-parameter tile
], ids=lambda c: f"M{c[0]}-{c[1]}-state{int(c[6])}")
def test_subset_at_the_segment_limit(env, case):
    """As many segments as the engine accepts, each of 1 to 3 parameters."""
    fgd, torch = env
    M, dtype, s1, k1, s2, k2, state = case
    n = fgd.FGD_MAX_SUBSET_SEGMENTS
    P = 3 * n + 123
    print(f"[variants] subset of {n} segments {case}", flush=True)
    pa.run_case(fgd, torch, M, P, dtype, s1, k1, s2, k2, seed=47, mom_std=1e-3, mix1_state=state,
                subset=_dense_segments(n, seed=5))


def test_subset_cleared_equals_full(env):
    """Setting a subset and then clearing it gives the full-Mix2 step."""
    fgd, torch = env
    M, P, dtype = 8, 3079, "f32"
    ld = pa.aligned_ld(P)
    from synth import tensors

    tp, tl, v = tensors.numpy_inputs(M, P, ld=ld, dtype=dtype, mom_std=1e-3, seed=43)
    t1, t2 = pa.topo(G, M, 1), pa.topo(RING, M, 1)
    full = pa.run_engine(fgd, torch, M, P, ld, dtype, t1, t2, tp, tl, v)
    cleared = pa.run_engine(fgd, torch, M, P, ld, dtype, t1, t2, tp, tl, v, subset=[])
    for a, b in zip(full, cleared):
        assert np.array_equal(a, b)


def test_subset_needs_csr_mix2(env):
    fgd, torch = env
    M, P = 4, 1024
    dev = torch.device("cuda:0")
    tp = torch.zeros((M, P), dtype=torch.float32, device=dev)
    tl = torch.zeros_like(tp)
    v = torch.zeros_like(tp)
    eng = fgd.Engine(M, P, P, "f32", device=0)
    try:
        eng.set_topology("mix1", "global")
        eng.set_topology("mix2", "global")
        eng.set_mix2_subset([(0, 10)])
        with pytest.raises(fgd.FgdError) as ei:
            eng.outer_step(tp, tl, v)
        assert ei.value.status == fgd.FGD_ERR_UNSUPPORTED
    finally:
        eng.close()


def _random_case(i):
    """A seeded random configuration: worker count, size, storage, mixing kinds
    and rounds, masks and reweighting, optimizer form, state mix, subset."""
    rng = np.random.default_rng(1000 + i)
    M = int(rng.choice([1, 2, 3, 4, 5, 7, 8, 9, 12, 16, 17, 24, 32, 33, 48, 64]))
    P = int(rng.integers(1, 6000))
    dtype = str(rng.choice(["f32", "bf16"]))

    def spec():
        c = rng.integers(0, 6)
        if c == 0:
            return ID, 0
        if c == 1:
            return G, 1
        if c == 2:
            return ("complete",), int(rng.integers(1, 3))
        if c == 3:
            return ("er_mh", float(rng.uniform(0.1, 0.9)), float(rng.uniform(0, 0.5))), int(rng.integers(1, 4))
        if c == 4:
            return ("ring_self", float(rng.uniform(0, 0.5))), int(rng.integers(1, 4))
        return ("matching",), int(rng.integers(1, 3))

    (s1, k1), (s2, k2) = spec(), spec()
    if M < 3 and s2[0] in ("ring_self",):
        s2, k2 = G, 1
    if M < 3 and s1[0] in ("ring_self",):
        s1, k1 = G, 1
    subset = None
    csr2 = s2[0] not in ("identity", "global")
    if csr2 and rng.random() < 0.5:
        cuts = np.sort(rng.choice(np.arange(0, P + 1), size=min(P + 1, 2 * int(rng.integers(1, 4))), replace=False))
        subset = [(int(a), int(b)) for a, b in zip(cuts[0::2], cuts[1::2]) if b > a] or None
    return dict(M=M, P=P, dtype=dtype, s1=s1, k1=k1, s2=s2, k2=k2, nesterov=bool(rng.random() < 0.7),
                state=bool(rng.random() < 0.3), subset=subset)


@pytest.mark.parametrize("i", range(200))
def test_random_configurations(env, i):
    fgd, torch = env
    c = _random_case(i)
    print(f"[variants] random case {i}: {c}", flush=True)
    pa.run_case(fgd, torch, c["M"], c["P"], c["dtype"], c["s1"], c["k1"], c["s2"], c["k2"], seed=100 + i,
                mom_std=1e-3, nesterov=c["nesterov"], mix1_state=c["state"], subset=c["subset"])
