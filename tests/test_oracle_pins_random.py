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


@settings(max_examples=80, deadline=None)
@given(K=st.integers(2, 40), k_frac=st.floats(0.0, 1.0), scale=st.sampled_from([0.1, 1.0, 8.0, 200.0]),
       n_masked=st.integers(0, 5), tie_levels=st.integers(0, 3), seed=st.integers(0, 2 ** 31 - 1))
def test_js_distance_equals_rel_entr_over_an_independently_sorted_top_k(K, k_frac, scale, n_masked, tie_levels, seed):
    """d = sqrt(JS / ln 2) with JS = 1/2 sum_{i in T} p_i log(p_i / m_i)
    + 1/2 sum_{i in T} q_i log(q_i / m_i), m = (p + q) / 2, p and q the
    full-vocabulary softmax, T the k largest averaged-model logits with lower
    index first on ties (Sec. 4.4; App. D.2).  Built here from scipy's
    softmax and rel_entr (0 log 0 = 0) and a Python sort."""
    import math

    from scipy.special import rel_entr, softmax

    from oracle import js as ojs

    rng = np.random.default_rng(seed)
    za = rng.standard_normal(K) * scale
    zw = za + rng.standard_normal(K) * scale * 0.3
    if tie_levels:  # snap some logits onto a few shared values
        levels = rng.standard_normal(tie_levels) * scale
        for arr in (za, zw):
            pick = rng.random(K) < 0.4
            arr[pick] = levels[rng.integers(0, tie_levels, pick.sum())]
    for arr in (za, zw):  # masked tokens (logit -inf), keeping one finite logit
        idx = rng.permutation(K)[:min(n_masked, K - 1)]
        arr[idx] = -np.inf
    k = max(1, int(round(k_frac * K)))
    p, q = softmax(zw), softmax(za)
    top = sorted(range(K), key=lambda i: (-za[i], i))[:k]
    m = 0.5 * (p + q)
    js = 0.0
    for i in sorted(top):
        js += 0.5 * float(rel_entr(p[i], m[i])) + 0.5 * float(rel_entr(q[i], m[i]))
    want = math.sqrt(max(js, 0.0) / math.log(2.0))
    got = ojs.js_distance_token(zw, za, k)
    assert abs(got - want) <= 1e-12 + 1e-9 * want, (got, want)
    assert list(ojs.top_k_indices(za, k)) == sorted(top)
