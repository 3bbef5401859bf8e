"""The five outer-step workloads and the step variants measured on the largest, as data.

Each entry states the worker count M, the parameter count P per worker, the
storage dtype, the input distributions, the (Mix1, Mix2) topologies and rounds,
and the seed.  Topology entries name a structure from ``synth.graphs`` and how
its weights are obtained:

    ("global",)                          exact mean over all workers
    ("identity",)                        no mixing
    ("ring", "given")                    ring, 1/3 on self and each neighbour
    ("exp", "given")                     directed exponential graph, hops 1,2,4,8, 1/5 each
    ("ring", "metropolis", p_drop)       ring, per-round undirected edge drops, Metropolis weights
    ("regular", "metropolis", d)         seeded random d-regular graph, Metropolis weights

The M=64 random 4-regular structure is stored as a committed fixture
(tests/golden/regular4_m64_seed0.json) so the workload does not depend on
numpy's generator across versions.
"""

from __future__ import annotations

import json
import os

import numpy as np

from . import graphs

_HERE = os.path.dirname(os.path.abspath(__file__))
_GOLDEN = os.path.join(os.path.dirname(_HERE), "tests", "golden")

OUTER_LR = 0.7
MOMENTUM = 0.9

WORKLOADS = {
    "tiny_m4_p1m_f32": dict(
        M=4, P=1_048_576, dtype="f32", prev_std=0.02, drift_std=1e-3, mom_std=0.0, seed=0,
        mix1=("global",), k1=1, mix2=("ring", "given"), k2=1),
    "m8_p150m_f32": dict(
        M=8, P=150_000_000, dtype="f32", prev_std=0.02, drift_std=1e-3, mom_std=1e-4, seed=0,
        mix1=("global",), k1=1, mix2=("ring", "given"), k2=1),
    "m16_p500m_f32": dict(
        M=16, P=500_000_000, dtype="f32", prev_std=0.02, drift_std=1e-3, mom_std=1e-4, seed=1,
        mix1=("global",), k1=1, mix2=("exp", "given"), k2=2),
    "m8_p1100m_bf16": dict(
        M=8, P=1_100_000_000, dtype="bf16", prev_std=0.02, drift_std=1e-3, mom_std=1e-4, seed=0,
        mix1=("global",), k1=1, mix2=("ring", "metropolis", 0.1), k2=1),
    "m64_p124m_f32": dict(
        M=64, P=124_000_000, dtype="f32", prev_std=0.02, drift_std=2e-3, mom_std=1e-4, seed=0,
        mix1=("regular", "metropolis", 4), k1=1, mix2=("regular", "metropolis", 4), k2=3),
}

# Step variants on the 8 x 1.1e9 bf16 workload (same inputs and topologies):
#   subset43   GlobalM1LocalM2-subset: Mix2 on 43% of the parameters, as two
#              blocks at the two ends of the flattened vector (the paper's
#              subset is the token embeddings and first two layers at the
#              front plus the LM head at the back, 43% of a 1.5B model)
#   m1s        GlobalM1SLocalM2: the momentum is averaged by Mix1 too
#   m1s_subset43  both
SUBSET43 = ((0.0, 0.33), (0.90, 1.0))
for _name, _extra in (("subset43", dict(subset=SUBSET43)), ("m1s", dict(mix1_state=True)),
                      ("m1s_subset43", dict(subset=SUBSET43, mix1_state=True))):
    WORKLOADS["m8_p1100m_bf16_" + _name] = dict(WORKLOADS["m8_p1100m_bf16"], **_extra)


def subset_segments(w):
    """[n][2] int64 Mix2 subset segments of a workload (None: Mix2 everywhere).
    Fractions of P are rounded down to multiples of 8 parameters."""
    if not w.get("subset"):
        return None
    P = w["P"]
    cut = lambda f: min(P, int(f * P) // 8 * 8)
    return np.array([(cut(a), cut(b) if b < 1.0 else P) for a, b in w["subset"]], dtype=np.int64)


def regular4_m64():
    """The committed seeded 4-regular structure on 64 workers (with diagonal)."""
    with open(os.path.join(_GOLDEN, "regular4_m64_seed0.json")) as f:
        d = json.load(f)
    return np.array(d["row_ptr"], dtype=np.int32), np.array(d["col_idx"], dtype=np.int32)


def topology(spec, M, rounds, seed, step=0):
    """Resolve a topology spec into keyword arguments for set_topology.

    Returns dict(kind, row_ptr, col_idx, weights, rounds, masks, reweight) where
    kind is "identity", "global" or "csr" and reweight is "none",
    "metropolis" or "self".  `step` selects the per-step mask draw for
    workloads whose masks change every outer step.
    """
    name = spec[0]
    if name == "identity" or rounds == 0:
        return dict(kind="identity", row_ptr=None, col_idx=None, weights=None, rounds=0, masks=None,
                    reweight="none")
    if name == "global":
        return dict(kind="global", row_ptr=None, col_idx=None, weights=None, rounds=1, masks=None,
                    reweight="none")
    if name == "ring" and spec[1] == "given":
        rp, ci, w = graphs.ring_weights(M)
        return dict(kind="csr", row_ptr=rp, col_idx=ci, weights=w, rounds=rounds, masks=None,
                    reweight="none")
    if name == "exp" and spec[1] == "given":
        rp, ci, w = graphs.exponential_weights(M)
        return dict(kind="csr", row_ptr=rp, col_idx=ci, weights=w, rounds=rounds, masks=None,
                    reweight="none")
    if name == "ring" and spec[1] == "metropolis":
        rp, ci = graphs.ring(M)
        masks = graphs.edge_drop_masks(rp, ci, rounds, spec[2], seed=seed * 1_000_003 + step)
        return dict(kind="csr", row_ptr=rp, col_idx=ci, weights=None, rounds=rounds, masks=masks,
                    reweight="metropolis")
    if name == "regular" and spec[1] == "metropolis":
        if M == 64 and spec[2] == 4:
            rp, ci = regular4_m64()
        else:
            rp, ci = graphs.random_regular(M, spec[2], seed)
        return dict(kind="csr", row_ptr=rp, col_idx=ci, weights=None, rounds=rounds, masks=None,
                    reweight="metropolis")
    raise ValueError(f"unknown topology spec {spec}")


def min_bytes_per_step(M, P, dtype):
    """Algorithmic minimum HBM bytes of one outer step: read theta_prev,
    theta_local and momentum, write theta_prev and momentum."""
    ep = 4 if dtype == "f32" else 2
    return M * P * (3 * ep + 2 * 4)
