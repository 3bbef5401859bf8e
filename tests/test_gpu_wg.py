"""GPU parity of the 64-worker worker-group step kernel against the oracle.

fgd_outer_step launches it for 64 workers on sparse CSR mixes (a lane holds
16 workers x 4 parameters); every case here checks that it did
(Engine.step_variant) and compares theta', v' and every consensus row with
the oracle (Sec. 3 mixing, Sec. 4.1 factored step, Appendix B Nesterov,
Sec. 4.4 / Appendix D.1 consensus): ragged and single-parameter tiles, grids
that stride over several tiles, the most unrolled rounds of both mixes,
padded tables (rows with fewer live entries than the widest), directed and
matching topologies, both storages, both optimizer forms.
"""

import numpy as np
import pytest

from tests import _parity as pa

pytestmark = pytest.mark.gpu

G = ("global",)
REG4 = ("regular", "metropolis", 4)
RING_MH = ("ring", "metropolis", 0.1)


@pytest.fixture(scope="module")
def env():
    import torch

    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    import paper_2606_22768_amd as fgd

    return fgd, torch


# (P, dtype, mix1, K1, mix2, K2)
CASES = [
    (775, "f32", REG4, 1, REG4, 3),             # three full tiles and a ragged one
    (256, "f32", REG4, 1, REG4, 3),             # exactly one tile
    (3, "f32", REG4, 1, REG4, 1),               # less than one lane vector
    (300_001, "f32", REG4, 1, REG4, 3),         # more tiles than blocks: each block strides
    (300_001, "bf16", REG4, 1, REG4, 3),
    (1029, "bf16", G, 1, REG4, 4),              # GlobalM1LocalM2 with the most Mix2 rounds
    (1029, "f32", REG4, 2, REG4, 4),            # the most rounds of both mixes
    (2051, "f32", G, 1, RING_MH, 3),            # per-round drops, padded tables
    (2051, "bf16", ("er_mh", 0.1, 0.2), 1, ("er_mh", 0.1, 0.2), 1),  # rows up to 15 entries, padded
    (2051, "f32", ("exp", "given"), 1, ("exp", "given"), 2),          # directed doubly-stochastic W
    (4101, "f32", ("matching",), 2, ("matching",), 4),                # random pairwise gossip
    (999, "bf16", ("ring_self", 0.3), 2, ("ring_self", 0.3), 3),      # self reweighting
]


def _ids(c):
    return f"P{c[0]}-{c[1]}-{c[2][0]}{c[3]}-{c[4][0]}{c[5]}"


@pytest.mark.parametrize("case", CASES, ids=_ids)
def test_worker_group_step(env, case):
    fgd, torch = env
    P, dtype, s1, k1, s2, k2 = case
    print(f"[wg] {case}", flush=True)
    pa.run_case(fgd, torch, 64, P, dtype, s1, k1, s2, k2, seed=7)
    assert pa.last_variant == "worker-groups"


@pytest.mark.parametrize("nesterov, lr, mu, with_cd", [(False, 0.7, 0.9, True), (True, 1.0, 0.5, False),
                                                       (True, 0.3, 0.0, True)])
def test_worker_group_optimizer_forms(env, nesterov, lr, mu, with_cd):
    fgd, torch = env
    print(f"[wg] nesterov={nesterov} lr={lr} mu={mu} cd={with_cd}", flush=True)
    pa.run_case(fgd, torch, 64, 2 * 1024 + 77, "f32", REG4, 1, REG4, 3, seed=8, nesterov=nesterov, lr=lr, mu=mu,
                with_cd=with_cd)
    assert pa.last_variant == "worker-groups"


def test_worker_group_padded_row_stride(env):
    """ld well above P: the padding columns are never written."""
    fgd, torch = env
    print("[wg] ld > P", flush=True)
    pa.run_case(fgd, torch, 64, 1000, "bf16", REG4, 1, REG4, 2, ld=1000 + 136, seed=9)
    assert pa.last_variant == "worker-groups"


def _random_case(seed):
    rng = np.random.default_rng(seed)
    specs = [REG4, RING_MH, ("er_mh", float(rng.uniform(0.03, 0.1)), float(rng.uniform(0, 0.4))),
             ("exp", "given"), ("matching",), ("ring_self", float(rng.uniform(0, 0.5)))]
    s2 = specs[int(rng.integers(0, len(specs)))]
    s1 = G if rng.random() < 0.4 else specs[int(rng.integers(0, len(specs)))]
    k1 = 1 if s1 == G else int(rng.integers(1, 3))
    k2 = int(rng.integers(1, 5))
    P = int(rng.choice([int(rng.integers(1, 600)), int(rng.integers(600, 20_000)), int(rng.integers(2e5, 4e5))]))
    return dict(P=P, dtype=["f32", "bf16"][int(rng.integers(0, 2))], s1=s1, k1=k1, s2=s2, k2=k2,
                nesterov=bool(rng.random() < 0.8), seed=seed)


@pytest.mark.parametrize("i", range(40))
def test_worker_group_random_configurations(env, i):
    """Seeded random sparse topologies, rounds, sizes, storages and optimizer
    forms at 64 workers; those the worker-group kernel serves must match the
    oracle through it (the rest are still checked, on the other kernel)."""
    fgd, torch = env
    c = _random_case(9000 + i)
    print(f"[wg random] {c}", flush=True)
    pa.run_case(fgd, torch, 64, c["P"], c["dtype"], c["s1"], c["k1"], c["s2"], c["k2"], seed=c["seed"],
                nesterov=c["nesterov"])
