"""Randomised pins of the oracle's whole step (CPU).

For random small undirected graphs with random per-round edge drops, the
oracle's step (Metropolis reweighting done inside the oracle) is compared with
the step written as dense float64 matrix products (Sec. 3 mixing operator:
row m of W pulls the columns listed in row m; Sec. 4.1 factored step; App. B
Nesterov form).  The paper fixes no weights for a graph with dropped links;
the rule taken here is Metropolis on the live graph of each round, computed in
this file from its definition: w_ij = 1 / (1 + max(d_i, d_j)) for a live edge
(d = live neighbours) and w_ii = 1 - sum of row i's other weights, in float64
and then rounded to float32.  This pins the oracle's CSR walk, masks, round
composition and weight rounding on many more shapes than the hand cases.
"""

import numpy as np
import pytest
from hypothesis import given, settings
from hypothesis import strategies as st

import oracle


def _random_graph(rng, M, p_edge):
    A = np.triu(rng.random((M, M)) < p_edge, 1)
    A = A | A.T
    row_ptr, col_idx = [0], []
    for i in range(M):
        cols = sorted(set(np.nonzero(A[i])[0].tolist()) | {i})
        col_idx += cols
        row_ptr.append(len(col_idx))
    return np.array(row_ptr, np.int32), np.array(col_idx, np.int32)


def _random_masks(rng, row_ptr, col_idx, rounds, p_drop):
    """Per round, each undirected edge dropped with probability p_drop
    (both directions together); the diagonal stays live."""
    M = len(row_ptr) - 1
    masks = np.ones((rounds, len(col_idx)), np.uint8)
    for k in range(rounds):
        drop = np.triu(rng.random((M, M)) < p_drop, 1)
        drop = drop | drop.T
        for i in range(M):
            for e in range(row_ptr[i], row_ptr[i + 1]):
                j = col_idx[e]
                if j != i and drop[i, j]:
                    masks[k, e] = 0
    return masks


def _metropolis_dense(row_ptr, col_idx, mask):
    """Dense float32 W of one round from the definition (see module doc)."""
    M = len(row_ptr) - 1
    live = np.zeros((M, M), bool)
    for i in range(M):
        for e in range(row_ptr[i], row_ptr[i + 1]):
            j = col_idx[e]
            if j != i and (mask is None or mask[e]):
                live[i, j] = True
    deg = live.sum(axis=1)
    W = np.zeros((M, M), np.float64)
    for i in range(M):
        off = 0.0
        for j in range(M):  # ascending j
            if live[i, j]:
                w = 1.0 / (1.0 + max(deg[i], deg[j]))
                W[i, j] = np.float32(w)
                off += w
        W[i, i] = np.float32(1.0 - off)
    return W


@settings(max_examples=60, deadline=None)
@given(M=st.integers(1, 9), P=st.integers(1, 24), k1=st.integers(0, 3), k2=st.integers(0, 3),
       p_edge=st.floats(0.0, 1.0), p_drop=st.floats(0.0, 0.6), nesterov=st.booleans(),
       seed=st.integers(0, 2 ** 31 - 1))
def test_step_equals_dense_products_on_random_graphs(M, P, k1, k2, p_edge, p_drop, nesterov, seed):
    rng = np.random.default_rng(seed)
    row_ptr, col_idx = _random_graph(rng, M, p_edge)
    m1 = _random_masks(rng, row_ptr, col_idx, max(k1, 1), p_drop)[:k1]
    m2 = _random_masks(rng, row_ptr, col_idx, max(k2, 1), p_drop)[:k2]
    tp = (rng.standard_normal((M, P)) * 0.02).astype(np.float32)
    tl = (tp + rng.standard_normal((M, P)) * 1e-3).astype(np.float32)
    v = (rng.standard_normal((M, P)) * 1e-4).astype(np.float32)
    lr, mu = np.float32(rng.uniform(0.1, 1.0)), np.float32(rng.uniform(0.0, 0.95))
    mix1 = oracle.Mix("csr", row_ptr, col_idx, None, rounds=k1, masks=m1 if k1 else None, reweight="metropolis")
    mix2 = oracle.Mix("csr", row_ptr, col_idx, None, rounds=k2, masks=m2 if k2 else None, reweight="metropolis")
    out_t, out_v, cd = oracle.outer_step(tp, tl, v, mix1, mix2, lr=float(lr), mu=float(mu), nesterov=nesterov)

    x = tp.astype(np.float64)
    for k in range(k1):
        x = _metropolis_dense(row_ptr, col_idx, m1[k]) @ x
    g = tp.astype(np.float64) - tl.astype(np.float64)
    gs = [g]
    for k in range(k2):
        g = _metropolis_dense(row_ptr, col_idx, m2[k]) @ g
        gs.append(g)
    vn = float(mu) * v.astype(np.float64) + g
    step = g + float(mu) * vn if nesterov else vn
    want_t = x - float(lr) * step
    scale = max(np.abs(want_t).max(), 1e-30)
    np.testing.assert_allclose(out_t, want_t, rtol=0, atol=scale * 2.4e-7)
    np.testing.assert_allclose(out_v, vn, rtol=0, atol=max(np.abs(vn).max(), 1e-30) * 2.4e-7)
    # Consensus rows of the Mix2 intermediates: S_m = sum_p (u_m - mean)^2.
    for r, u in enumerate(gs):
        want_cd = ((u - u.mean(axis=0)) ** 2).sum(axis=1)
        np.testing.assert_allclose(cd[r], want_cd, rtol=1e-9, atol=1e-18)
