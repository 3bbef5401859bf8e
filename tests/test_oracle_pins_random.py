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
    got = ojs.js_distance_token(zw, za, k)
    # Compared as JS = d^2 ln 2: the square root would amplify the rounding
    # of a JS near 0 (d ~ 1e-6 turns an error of 1e-17 in JS into 3e-12 in
    # d).  The two sums of at most K terms, each below 1 in magnitude, differ
    # in rounding by at most about K * 2^-52 absolute.
    got_js = got * got * math.log(2.0)
    assert abs(got_js - max(js, 0.0)) <= K * 2.0 ** -52 + 1e-12 * js, (got_js, js)
    assert list(ojs.top_k_indices(za, k)) == sorted(top)


def _random_segments(rng, P):
    """Ascending, disjoint, non-empty half-open segments inside [0, P)."""
    cuts = np.sort(rng.choice(np.arange(P + 1), size=min(P + 1, 2 * int(rng.integers(1, 4))), replace=False))
    segs = [(int(cuts[i]), int(cuts[i + 1])) for i in range(0, len(cuts) - 1, 2) if cuts[i + 1] > cuts[i]]
    return segs or [(0, P)]


def _dense_rounds(row_ptr, col_idx, masks, kind, M, rounds):
    """Per-round dense matrices of a Mix slot (identity: none; global: one J)."""
    if kind == "identity":
        return []
    if kind == "global":
        return [np.full((M, M), 1.0 / M)]
    return [_metropolis_dense(row_ptr, col_idx, masks[k]) for k in range(rounds)]


def _apply(Ws, u, cols=None):
    """Rounds applied in order; with cols, only on those columns (identity
    elsewhere).  Returns every intermediate, input first."""
    out = [u]
    for W in Ws:
        nxt = out[-1].copy()
        if cols is None:
            nxt = W @ out[-1]
        else:
            nxt[:, cols] = W @ out[-1][:, cols]
        out.append(nxt)
    return out


def _S(u):
    return ((u - u.mean(axis=0)) ** 2).sum(axis=1)


@settings(max_examples=60, deadline=None)
@given(M=st.integers(2, 8), P=st.integers(1, 20), k1=st.integers(1, 2), k2=st.integers(1, 3),
       kind1=st.sampled_from(["csr", "global", "identity"]), kind2=st.sampled_from(["csr", "identity"]),
       nesterov=st.booleans(), state=st.booleans(), use_subset=st.booleans(), write_local=st.booleans(),
       seed=st.integers(0, 2 ** 31 - 1))
def test_variants_and_split_halves_equal_dense_products(M, P, k1, k2, kind1, kind2, nesterov, state, use_subset,
                                                         write_local, seed):
    """Plain momentum (App. B without the Nesterov term), Mix1 on the state
    (App. B, GlobalM1S), a Mix2 subset (Sec. 4.1, App. C: Mix2 on the listed
    columns, identity elsewhere, consensus over every column) and the two
    halves of split execution (App. A, Alg. 1) against dense float64 products
    on random graphs with link drops."""
    rng = np.random.default_rng(seed)
    row_ptr, col_idx = _random_graph(rng, M, 0.6)
    m1 = _random_masks(rng, row_ptr, col_idx, k1, 0.3)
    m2 = _random_masks(rng, row_ptr, col_idx, k2, 0.3)
    if kind2 != "csr":
        use_subset = False  # a subset needs a table Mix2
    segs = _random_segments(rng, P) if use_subset else None
    cols = None if segs is None else np.concatenate([np.arange(b, e) for b, e in segs])
    tp = (rng.standard_normal((M, P)) * 0.02).astype(np.float32)
    tl = (tp + rng.standard_normal((M, P)) * 1e-3).astype(np.float32)
    v = (rng.standard_normal((M, P)) * 1e-4).astype(np.float32)
    lr, mu = float(np.float32(rng.uniform(0.1, 1.0))), float(np.float32(rng.uniform(0.0, 0.95)))

    def mix(kind, masks, rounds):
        if kind == "csr":
            return oracle.Mix("csr", row_ptr, col_idx, None, rounds=rounds, masks=masks, reweight="metropolis")
        return oracle.Mix(kind)

    mix1, mix2 = mix(kind1, m1, k1), mix(kind2, m2, k2)
    W1 = _dense_rounds(row_ptr, col_idx, m1, kind1, M, k1)
    W2 = _dense_rounds(row_ptr, col_idx, m2, kind2, M, k2)

    def check(got, want, what):
        tol = max(np.abs(want).max(), 1e-30) * 2.4e-7
        np.testing.assert_allclose(got, want, rtol=0, atol=tol, err_msg=what)

    def check_cd(got, rows, what):
        for r, u in enumerate(rows):
            np.testing.assert_allclose(got[r], _S(u), rtol=1e-9, atol=1e-18, err_msg=f"{what} row {r}")

    def optimizer(x, g, vin):
        vn = mu * vin + g
        return x - lr * (g + mu * vn if nesterov else vn), vn

    g_rows = _apply(W2, tp.astype(np.float64) - tl.astype(np.float64), cols)
    v_in = _apply(W1, v.astype(np.float64))[-1] if state else v.astype(np.float64)

    # Fused step.
    x_rows = _apply(W1, tp.astype(np.float64))
    want_t, want_v = optimizer(x_rows[-1], g_rows[-1], v_in)
    got_t, got_v, got_cd = oracle.outer_step(tp, tl, v, mix1, mix2, lr=lr, mu=mu, nesterov=nesterov,
                                             mix1_state=state, subset=segs)
    check(got_t, want_t, "theta'")
    check(got_v, want_v, "v'")
    check_cd(got_cd, g_rows + x_rows + [got_t.astype(np.float64)], "fused consensus")

    # Split halves: the Mix1 half stores x in float32; the blocking half reads it.
    x_st, v_st, cd1 = oracle.mix1_split(tp, mix1, mom=v, mix1_state=state)
    check(x_st, x_rows[-1], "stored x")
    check_cd(cd1, x_rows, "Mix1-half consensus")
    if state:
        check(v_st, v_in, "mixed state")
    vb = v_st if state else v
    want_t2, want_v2 = optimizer(x_st.astype(np.float64), g_rows[-1], vb.astype(np.float64))
    got_t2, got_tl2, got_v2, cd2 = oracle.outer_blocking(x_st, tp, tl, vb, mix2, lr=lr, mu=mu, nesterov=nesterov,
                                                         subset=segs, write_local=write_local)
    check(got_t2, want_t2, "blocking theta'")
    check(got_v2, want_v2, "blocking v'")
    assert np.array_equal(got_tl2, got_t2 if write_local else tl)
    check_cd(cd2, g_rows + [got_t2.astype(np.float64)], "blocking consensus")
