"""Pins for the CPU oracle: each test fixes part of it against something other
than itself -- a library routine, a closed form from the paper, an invariant
of doubly-stochastic mixing, brute force on tiny inputs or exact rationals.

Runs on the CPU only.
"""

import json
import os
from fractions import Fraction

import numpy as np
import pytest
import scipy.sparse
import torch

import oracle
from synth import graphs, tensors

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
LR, MU = np.float32(0.7), np.float32(0.9)


def dense_W(row_ptr, col_idx, w):
    """Dense mixing matrix from CSR with scipy (row m, column j = weight of j in m's mix)."""
    M = len(row_ptr) - 1
    return scipy.sparse.csr_matrix((np.asarray(w, np.float64), col_idx, row_ptr), shape=(M, M)).toarray()


def f32(x):
    return np.float32(x)


# ----------------------------------------------------------------- Nesterov

@pytest.mark.parametrize("mix1,mix2", [("identity", "identity"), ("global", "global"), ("identity", "csr1")])
def test_nesterov_m1_matches_torch_sgd(mix1, mix2):
    """M=1: every mix is the identity and the step is torch's SGD with Nesterov
    momentum (Appendix B gives PyTorch's implementation form), gradient
    theta_prev - theta_local, momentum buffer preloaded with v."""
    P = 4099
    tp, tl, v = tensors.numpy_inputs(1, P, mom_std=1e-4, seed=3)
    m1 = oracle.Mix(mix1)
    if mix2 == "csr1":
        rp, ci, w = graphs.identity(1)
        m2 = oracle.Mix("csr", rp, ci, w, rounds=2)
    else:
        m2 = oracle.Mix(mix2)
    out_t, out_v, _ = oracle.outer_step(tp, tl, v, m1, m2, lr=LR, mu=MU)

    p = torch.nn.Parameter(torch.from_numpy(tp[0].astype(np.float64)))
    opt = torch.optim.SGD([p], lr=float(LR), momentum=float(MU), nesterov=True)
    p.grad = torch.from_numpy((tp[0].astype(np.float64) - tl[0].astype(np.float64)))
    opt.state[p]["momentum_buffer"] = torch.from_numpy(v[0].astype(np.float64)).clone()
    opt.step()
    want_t = p.detach().numpy()
    want_v = opt.state[p]["momentum_buffer"].numpy()
    # torch may fuse multiply-adds in double; agreement is to the float32 rounding.
    np.testing.assert_allclose(out_t[0], want_t, rtol=0, atol=np.abs(want_t).max() * 2 ** -23)
    np.testing.assert_allclose(out_v[0], want_v, rtol=0, atol=np.abs(want_v).max() * 2 ** -23)


def test_nesterov_expanded_form():
    """The two-line form equals the expanded form x - lr((1+mu) g + mu^2 v)
    (Appendix B), evaluated here independently in numpy double precision."""
    P = 2000
    tp, tl, v = tensors.numpy_inputs(1, P, mom_std=1e-3, seed=5)
    out_t, out_v, _ = oracle.outer_step(tp, tl, v, oracle.Mix("identity"), oracle.Mix("identity"))
    g = tp[0].astype(np.float64) - tl[0].astype(np.float64)
    mu, lr = float(MU), float(LR)
    want = tp[0].astype(np.float64) - lr * ((1 + mu) * g + mu * mu * v[0].astype(np.float64))
    np.testing.assert_allclose(out_t[0], want, rtol=0, atol=np.abs(want).max() * 2e-7)
    np.testing.assert_allclose(out_v[0], mu * v[0].astype(np.float64) + g, rtol=0,
                               atol=np.abs(out_v).max() * 2e-7)


# ------------------------------------------------------- DiLoCo reduction

@pytest.mark.parametrize("mix1", ["identity", "global"])
def test_diloco_reduction(mix1):
    """Equal theta_prev and v on all workers with a global Mix2 is DiLoCo's step
    (Sec. 3 DiLoCo equations; Appendix A configuration table: DiLoCo =
    identity Mix1, global Mix2): every worker gets Nesterov on the mean
    outer gradient, here via torch's SGD."""
    M, P = 5, 777
    rng = np.random.default_rng(11)
    base = (rng.standard_normal(P) * 0.02).astype(np.float32)
    tp = np.tile(base, (M, 1))
    tl = (tp + rng.standard_normal((M, P)).astype(np.float32) * np.float32(1e-3)).astype(np.float32)
    vb = (rng.standard_normal(P) * 1e-4).astype(np.float32)
    v = np.tile(vb, (M, 1))
    out_t, out_v, cd = oracle.outer_step(tp, tl, v, oracle.Mix(mix1), oracle.Mix("global"))

    gbar = (tp.astype(np.float64) - tl.astype(np.float64)).mean(axis=0)
    p = torch.nn.Parameter(torch.from_numpy(base.astype(np.float64)))
    opt = torch.optim.SGD([p], lr=float(LR), momentum=float(MU), nesterov=True)
    p.grad = torch.from_numpy(gbar)
    opt.state[p]["momentum_buffer"] = torch.from_numpy(vb.astype(np.float64)).clone()
    opt.step()
    want = p.detach().numpy()
    for m in range(M):
        np.testing.assert_allclose(out_t[m], want, rtol=0, atol=np.abs(want).max() * 2 ** -22)
    # Exact consensus after the step: every worker stores the same value.
    assert np.all(out_t == out_t[0])
    assert np.all(cd[-1] == 0.0)


# ------------------------------------------------- factored form, plain SGD

@pytest.mark.parametrize("topo", ["ring", "exp16", "complete"])
def test_plain_sgd_factored_form(topo):
    """With lr=1 and mu=0 the update is z' = Mix1(z) + Mix2(Delta), Delta =
    theta_local - theta_prev (Sec. 4.1 factored formulation; the outer
    optimizer receives -Delta-hat).  Mixes are evaluated as dense matrix
    products built by scipy from the CSR, which also fixes the orientation
    (row m pulls the columns listed in row m) on the directed exponential
    graph."""
    if topo == "ring":
        M = 6
        rp, ci, w = graphs.ring_weights(M)
        rp1, ci1, w1 = graphs.complete_weights(M)
    elif topo == "exp16":
        M = 16
        rp, ci, w = graphs.exponential_weights(M)
        rp1, ci1, w1 = graphs.ring_weights(M)
    else:
        M = 4
        rp, ci, w = graphs.complete_weights(M)
        rp1, ci1, w1 = graphs.exponential_weights(M, hops=(1,))
    P = 513
    tp, tl, v = tensors.numpy_inputs(M, P, mom_std=0.0, seed=7)
    mix1 = oracle.Mix("csr", rp1, ci1, w1, rounds=2)
    mix2 = oracle.Mix("csr", rp, ci, w, rounds=1)
    out_t, out_v, _ = oracle.outer_step(tp, tl, v, mix1, mix2, lr=1.0, mu=0.0)
    W1, W2 = dense_W(rp1, ci1, w1), dense_W(rp, ci, w)
    X = tp.astype(np.float64)
    delta = tl.astype(np.float64) - tp.astype(np.float64)
    want = W1 @ (W1 @ X) + W2 @ delta
    np.testing.assert_allclose(out_t, want, rtol=0, atol=np.abs(want).max() * 2e-7)
    np.testing.assert_allclose(out_v, -(W2 @ delta), rtol=0, atol=np.abs(delta).max() * 2e-7)


# -------------------------------------------------- doubly stochastic mixing

def _mixes_for_invariants():
    out = []
    rp, ci, w = graphs.ring_weights(8)
    out.append(("ring8_given", 8, oracle.Mix("csr", rp, ci, w, rounds=3)))
    rp, ci, w = graphs.exponential_weights(16)
    out.append(("exp16_given", 16, oracle.Mix("csr", rp, ci, w, rounds=2)))
    rp, ci = graphs.ring(8)
    masks = graphs.edge_drop_masks(rp, ci, 3, 0.3, seed=4)
    out.append(("ring8_mh_masks", 8, oracle.Mix("csr", rp, ci, None, rounds=3, masks=masks,
                                                reweight="metropolis")))
    rp, ci, w = graphs.ring_weights(8)
    out.append(("ring8_self_masks", 8, oracle.Mix("csr", rp, ci, w, rounds=3, masks=masks, reweight="self")))
    rp, ci = graphs.random_regular(12, 4, seed=2)
    out.append(("reg12_mh", 12, oracle.Mix("csr", rp, ci, None, rounds=2, reweight="metropolis")))
    out.append(("global", 7, oracle.Mix("global")))
    return out


@pytest.mark.parametrize("name,M,mix", _mixes_for_invariants(), ids=lambda x: x if isinstance(x, str) else "")
def test_mix_preserves_worker_mean(name, M, mix):
    """A doubly-stochastic W keeps the worker mean (Sec. 3: W symmetric and
    doubly stochastic).  With float32 weights the column sums are 1 to
    within a few float32 ulps, hence the tolerance."""
    rng = np.random.default_rng(1)
    X = rng.standard_normal((M, 300))
    Y, _ = oracle.mix_apply(mix, X)
    np.testing.assert_allclose(Y.mean(axis=0), X.mean(axis=0), rtol=0, atol=1e-6 * np.abs(X).max())


@pytest.mark.parametrize("name,M,mix", _mixes_for_invariants(), ids=lambda x: x if isinstance(x, str) else "")
def test_whole_step_mean_is_one_nesterov_step(name, M, mix):
    """Rearranged DiLoCo (Sec. 4.2): the outer step is linear, so with
    doubly-stochastic mixes the worker mean of the result is one Nesterov step
    on the worker means of theta_prev, the outer gradient and v."""
    P = 400
    tp, tl, v = tensors.numpy_inputs(M, P, mom_std=1e-4, seed=9)
    rp, ci, w = graphs.complete_weights(M)
    for mix1 in (oracle.Mix("global"), oracle.Mix("csr", rp, ci, w, rounds=1), mix):
        out_t, out_v, _ = oracle.outer_step(tp, tl, v, mix1, mix)
        xb = tp.astype(np.float64).mean(0)
        gb = (tp.astype(np.float64) - tl.astype(np.float64)).mean(0)
        vb = v.astype(np.float64).mean(0)
        vn = float(MU) * vb + gb
        want = xb - float(LR) * (gb + float(MU) * vn)
        np.testing.assert_allclose(out_t.astype(np.float64).mean(0), want, rtol=0,
                                   atol=2e-6 * np.abs(tp).max())
        np.testing.assert_allclose(out_v.astype(np.float64).mean(0), vn, rtol=0, atol=2e-6 * np.abs(vn).max())


def test_superposition():
    """The step is linear in (theta_prev, theta_local, v) jointly (Sec. 4.2):
    step(A + B) = step(A) + step(B) up to float32 output rounding, and scaling
    all inputs by 2 scales every output by exactly 2."""
    M, P = 8, 300
    rp, ci = graphs.ring(M)
    masks = graphs.edge_drop_masks(rp, ci, 2, 0.2, seed=8)
    mix2 = oracle.Mix("csr", rp, ci, None, rounds=2, masks=masks, reweight="metropolis")
    mix1 = oracle.Mix("global")
    rng = np.random.default_rng(12)

    def grid_inputs():
        # Integers times 2^-20: float32-exact, and so are their pairwise sums.
        return [(rng.integers(-2 ** 20, 2 ** 20, (M, P)) * 2.0 ** -20).astype(np.float32) for _ in range(3)]

    a, b = grid_inputs(), grid_inputs()
    s = [x + y for x, y in zip(a, b)]
    ra = oracle.outer_step(*a, mix1, mix2)
    rb = oracle.outer_step(*b, mix1, mix2)
    rs = oracle.outer_step(*s, mix1, mix2)
    for i in range(2):
        ref = ra[i].astype(np.float64) + rb[i].astype(np.float64)
        np.testing.assert_allclose(rs[i], ref, rtol=0, atol=4e-7 * np.abs(ref).max())
    two = [2 * x for x in a]
    r2 = oracle.outer_step(*two, mix1, mix2)
    np.testing.assert_array_equal(r2[0], 2 * ra[0])
    np.testing.assert_array_equal(r2[1], 2 * ra[1])
    np.testing.assert_array_equal(r2[2], 4 * ra[2])


# ---------------------------------------------------------------- contraction

def _lambda2(W):
    """Second-largest singular value of W (for symmetric W, the second-largest
    eigenvalue magnitude), by brute-force decomposition."""
    s = np.linalg.svd(W, compute_uv=False)
    return sorted(s)[-2]


@pytest.mark.parametrize("case", ["ring4", "ring8", "exp16", "reg12_mh", "ring8_masked"])
def test_contraction_bound_and_tightness(case):
    """Per round, S(WX) <= lambda_2(W)^2 S(X) (Sec. 3 contraction factor), with
    lambda_2 from a brute-force SVD of the dense W; equality for X aligned with
    the second singular vector.  Closed forms: ring-4 has lambda_2 = 1/3 and
    ring-8 (1 + 2 cos(pi/4))/3 (eigenvalues of the circulant with 1/3
    weights); the directed exponential graph on 16 has sigma_2 = 0.6."""
    masks = None
    if case.startswith("ring"):
        M = 4 if case == "ring4" else 8
        rp, ci, w = graphs.ring_weights(M)
        if case == "ring8_masked":
            masks = graphs.edge_drop_masks(rp, ci, 1, 0.3, seed=3)
            mix = oracle.Mix("csr", rp, ci, w, rounds=1, masks=masks, reweight="self")
            w = oracle.round_weights(rp, ci, w, masks[0], "self")
        else:
            mix = oracle.Mix("csr", rp, ci, w, rounds=1)
    elif case == "exp16":
        M = 16
        rp, ci, w = graphs.exponential_weights(M)
        mix = oracle.Mix("csr", rp, ci, w, rounds=1)
    else:
        M = 12
        rp, ci = graphs.random_regular(M, 4, seed=2)
        mix = oracle.Mix("csr", rp, ci, None, rounds=1, reweight="metropolis")
        w = oracle.round_weights(rp, ci, None, None, "metropolis")
    W = dense_W(rp, ci, w)
    lam = _lambda2(W)
    if case == "ring4":
        assert abs(lam - 1 / 3) < 1e-6
    if case == "ring8":
        assert abs(lam - (1 + 2 * np.cos(np.pi / 4)) / 3) < 1e-6
    if case == "exp16":
        assert abs(lam - 0.6) < 1e-6
    rng = np.random.default_rng(0)
    for _ in range(5):
        X = rng.standard_normal((M, 64))
        _, cd = oracle.mix_apply(mix, X)
        assert cd[1].sum() <= lam ** 2 * cd[0].sum() * (1 + 1e-6)
    # Tightness along the second right-singular vector (orthogonal to 1).
    U, s, Vt = np.linalg.svd(W)
    k = int(np.argsort(s)[-2])
    vec = Vt[k]
    X = np.outer(vec, rng.standard_normal(32))
    _, cd = oracle.mix_apply(mix, X)
    np.testing.assert_allclose(cd[1].sum(), lam ** 2 * cd[0].sum(), rtol=1e-6)


def test_global_and_identity_contraction():
    """Global averaging has contraction 0, identity 1 (Sec. 3)."""
    rng = np.random.default_rng(3)
    X = rng.standard_normal((6, 50))
    _, cd = oracle.mix_apply(oracle.Mix("global"), X)
    # The mean of M equal doubles can differ from them in the last bit only.
    assert cd[0].sum() > 0 and cd[1].sum() <= 1e-28 * cd[0].sum()
    rp, ci, w = graphs.identity(6)
    _, cd = oracle.mix_apply(oracle.Mix("csr", rp, ci, w, rounds=1), X)
    np.testing.assert_array_equal(cd[1], cd[0])


@pytest.mark.parametrize("M", [4, 6, 8])
def test_pairwise_gossip_expected_contraction(M):
    """Averaging over every perfect matching, random pairwise gossip contracts
    the squared distance to the mean by exactly (M-2)/(2(M-1)) (Sec. 3).
    Pairs are expressed as a complete structure masked to the matching with
    Metropolis weights (1/2 on self and partner)."""
    rp, ci = graphs.complete(M)
    matchings = graphs.all_perfect_matchings(M)
    assert len(matchings) == {4: 3, 6: 15, 8: 105}[M]
    rng = np.random.default_rng(M)
    X = rng.standard_normal((M, 40))
    ratios = []
    for mt in matchings:
        masks = graphs.masks_from_live_edges(rp, ci, [mt])
        mix = oracle.Mix("csr", rp, ci, None, rounds=1, masks=masks, reweight="metropolis")
        _, cd = oracle.mix_apply(mix, X)
        ratios.append(cd[1].sum() / cd[0].sum())
    np.testing.assert_allclose(np.mean(ratios), (M - 2) / (2 * (M - 1)), rtol=1e-12)


# ------------------------------------------------------- consensus distance

@pytest.mark.parametrize("M", [1, 2, 5, 9])
def test_consensus_pairwise_identity(M):
    """(1/M^2) sum_{m,s} ||u_m - u_s||^2 = (2/M) sum_m S_m: the pairwise
    disagreement of Appendix E against the mean-deviation form of Sec. 4.4 /
    Appendix D.1, by brute force."""
    rng = np.random.default_rng(M)
    U = rng.standard_normal((M, 37)).astype(np.float32)
    S = oracle.consensus(U)
    Ud = U.astype(np.float64)
    pair = sum(((Ud[m] - Ud[s]) ** 2).sum() for m in range(M) for s in range(M)) / M ** 2
    np.testing.assert_allclose(pair, 2.0 / M * S.sum(), rtol=1e-12, atol=1e-300)


def test_consensus_bf16_and_ld():
    """S_m reads bf16 storage exactly and ignores the padding beyond P."""
    M, P, ld = 3, 100, 128
    rng = np.random.default_rng(5)
    X = rng.standard_normal((M, ld)).astype(np.float32)
    b = tensors.f32_to_bf16_bits(X)
    S = oracle.consensus(b, P=P)
    Xd = tensors.bf16_bits_to_f32(b)[:, :P].astype(np.float64)
    want = ((Xd - Xd.mean(0)) ** 2).sum(1)
    np.testing.assert_allclose(S, want, rtol=1e-12)


def test_step_cd_rows():
    """The step reports S_m of g^0..g^K2, x^0..x^K1 and the stored theta'.
    Checked against numpy: g^0 = theta_prev - theta_local, x^0 = theta_prev,
    the global-mean row is zero, and the last row equals S_m of the output."""
    M, P = 6, 250
    tp, tl, v = tensors.numpy_inputs(M, P, seed=4)
    rp, ci, w = graphs.ring_weights(M)
    mix2 = oracle.Mix("csr", rp, ci, w, rounds=2)
    out_t, _, cd = oracle.outer_step(tp, tl, v, oracle.Mix("global"), mix2)
    assert cd.shape == (3 + 2 + 1, M)

    def S(u):
        u = u.astype(np.float64)
        return ((u - u.mean(0)) ** 2).sum(1)

    np.testing.assert_allclose(cd[0], S(tp.astype(np.float64) - tl), rtol=1e-12)
    np.testing.assert_allclose(cd[3], S(tp), rtol=1e-12)
    assert np.all(cd[4] == 0.0)
    np.testing.assert_allclose(cd[5], S(out_t), rtol=1e-12)
    W = dense_W(rp, ci, w)
    g0 = tp.astype(np.float64) - tl
    np.testing.assert_allclose(cd[1], S(W @ g0), rtol=1e-9)
    np.testing.assert_allclose(cd[2], S(W @ (W @ g0)), rtol=1e-9)


# ----------------------------------------------------------- mixing weights

def _golden_cases():
    with open(os.path.join(GOLDEN, "metropolis_cases.json")) as f:
        return json.load(f)["cases"]


@pytest.mark.parametrize("case", _golden_cases(), ids=lambda c: c["name"])
def test_metropolis_hand_cases(case):
    """Metropolis weights against hand-computed fractions (golden fixture)."""
    M = case["M"]
    row_ptr, col_idx = graphs._csr_from_rows(case["rows"])
    masks = graphs.masks_from_live_edges(row_ptr, col_idx, [case["live"]])
    w = oracle.round_weights(row_ptr, col_idx, None, masks[0], "metropolis")
    for i in range(M):
        for e in range(row_ptr[i], row_ptr[i + 1]):
            j = int(col_idx[e])
            want = np.float32(float(Fraction(case["weights"][f"{i},{j}"])))
            assert w[e] == want, (case["name"], i, j, w[e], want)


def test_self_reweight_hand_case():
    """Self reweighting: a dropped edge's weight moves to both endpoints'
    diagonal.  Ring-8, 1/3 weights, edge (0,1) dropped: w_00 = w_11 = 2/3."""
    rp, ci, w = graphs.ring_weights(8)
    live = [e for e in graphs.undirected_edges(rp, ci) if e != (0, 1)]
    masks = graphs.masks_from_live_edges(rp, ci, [live])
    out = oracle.round_weights(rp, ci, w, masks[0], "self")
    W = dense_W(rp, ci, out)
    assert W[0, 0] == np.float32(np.float64(np.float32(1 / 3)) * 2)
    assert W[0, 1] == 0 and W[1, 0] == 0
    assert W[2, 2] == np.float32(1 / 3)


def test_weights_reject_bad_input():
    rp, ci, w = graphs.ring_weights(4)
    masks = graphs.edge_drop_masks(rp, ci, 1, 0.5, seed=1)
    masks[0][:] = 1
    masks[0][1] = 0
    with pytest.raises(ValueError):
        oracle.round_weights(rp, ci, w, masks[0], "none")  # masks under NONE
    diag_mask = np.ones(len(ci), np.uint8)
    diag_mask[rp[0] + list(ci[rp[0]:rp[1]]).index(0)] = 0
    with pytest.raises(ValueError):
        oracle.round_weights(rp, ci, w, diag_mask, "metropolis")  # masked diagonal


def test_fully_masked_worker_is_identity_row():
    """A worker whose links all dropped keeps its own value (weight 1 on self)."""
    M = 5
    rp, ci = graphs.ring(M)
    live = [e for e in graphs.undirected_edges(rp, ci) if 2 not in e]
    masks = graphs.masks_from_live_edges(rp, ci, [live])
    mix = oracle.Mix("csr", rp, ci, None, rounds=1, masks=masks, reweight="metropolis")
    rng = np.random.default_rng(0)
    X = rng.standard_normal((M, 20))
    X[1, 3] = np.inf  # a dropped neighbour's non-finite value does not leak
    Y, _ = oracle.mix_apply(mix, X)
    np.testing.assert_array_equal(Y[2], X[2])


# ----------------------------------------------------------------------- bf16

def _bf16_exact(x: float) -> int:
    """Nearest bf16 to x with ties to even, by exact rational comparison."""
    if np.isnan(x):
        return None
    sign = 0x8000 if np.signbit(x) else 0
    fx = Fraction(abs(x))
    # Enumerate the two bf16 neighbours through float32 bit patterns.
    f32v = np.float32(abs(x)) if abs(x) < 3.4e38 else np.float32(np.inf)
    bits = int(np.array([f32v], dtype=np.float32).view(np.uint32)[0]) >> 16
    cands = [max(bits - 1, 0), bits, min(bits + 1, 0x7F80)]
    best = None
    for c in cands:
        val = np.array([c << 16], dtype=np.uint32).view(np.float32)[0]
        if np.isinf(val):
            # Overflow threshold: halfway between the largest finite bf16 and 2^128.
            d = Fraction(2) ** 128 - fx
        else:
            d = abs(Fraction(float(val)) - fx)
        key = (d, c & 1)
        if best is None or key < best[0]:
            best = (key, c)
    return best[1] | sign


def test_bf16_rounding_exact():
    """Direct double -> bf16 rounding against exact rational nearest-even,
    over random magnitudes, subnormals, ties and the overflow edge."""
    rng = np.random.default_rng(0)
    vals = list(rng.standard_normal(3000) * np.exp(rng.uniform(-100, 100, 3000)))
    vals += list(rng.standard_normal(500) * 1e-39)  # bf16 subnormal range
    # Exact ties: midpoints between consecutive bf16 values.
    for b in [0x3F80, 0x3F81, 0x4049, 0x0001, 0x0080, 0x7F7E]:
        lo = np.array([b << 16], dtype=np.uint32).view(np.float32)[0]
        hi = np.array([(b + 1) << 16], dtype=np.uint32).view(np.float32)[0]
        vals.append((float(lo) + float(hi)) / 2)
        vals.append(-(float(lo) + float(hi)) / 2)
    vals += [0.0, -0.0, 1.0, -2.5, 3.3895313892515355e38, 3.3961775292304e38, 1e300, -1e300]
    for x in vals:
        got = oracle.bf16_from_double(float(x))
        want = _bf16_exact(float(x))
        assert got == want, (x, hex(got), hex(want))
    assert oracle.bf16_from_double(float("nan")) & 0x7FC0 == 0x7FC0


def test_bf16_ties_to_even_by_hand():
    """1 + 2^-8 lies halfway between bf16 1.0 (0x3F80) and 1 + 2^-7 (0x3F81): even wins.
    1 + 3*2^-8 lies between 0x3F81 and 0x3F82: even (0x3F82) wins."""
    assert oracle.bf16_from_double(1 + 2 ** -8) == 0x3F80
    assert oracle.bf16_from_double(1 + 3 * 2 ** -8) == 0x3F82
    assert oracle.bf16_from_double(1 + 2 ** -8 + 2 ** -30) == 0x3F81


# --------------------------------------------------------------- edge cases

def test_empty_and_padding():
    """P = 0 is a no-op; entries beyond P in an [M][ld] row are never touched."""
    M, P, ld = 3, 10, 16
    tp, tl, v = tensors.numpy_inputs(M, P, ld=ld, seed=1)
    tp[:, P:] = 123.0
    v[:, P:] = -7.0
    rp, ci, w = graphs.ring_weights(M)
    out_t, out_v, _ = oracle.outer_step(tp, tl, v, oracle.Mix("global"), oracle.Mix("csr", rp, ci, w, 1), P=P)
    assert np.all(out_t[:, P:] == 123.0) and np.all(out_v[:, P:] == -7.0)
    out_t, out_v, cd = oracle.outer_step(tp, tl, v, oracle.Mix("global"), oracle.Mix("csr", rp, ci, w, 1), P=0)
    np.testing.assert_array_equal(out_t, tp)
    assert np.all(cd == 0)


def test_bf16_step_close_to_f32_step():
    """bf16 storage: the same step computed from bf16-exact inputs in float32
    storage, then rounded to bf16, differs by at most one bf16 ulp (double
    rounding through float32)."""
    M, P = 4, 3000
    tpb, tlb, v = tensors.numpy_inputs(M, P, dtype="bf16", seed=6)
    tpf, tlf = tensors.bf16_bits_to_f32(tpb), tensors.bf16_bits_to_f32(tlb)
    rp, ci, w = graphs.ring_weights(M)
    mix2 = oracle.Mix("csr", rp, ci, w, 1)
    ob, vb, _ = oracle.outer_step(tpb, tlb, v, oracle.Mix("global"), mix2)
    of, vf, _ = oracle.outer_step(tpf, tlf, v, oracle.Mix("global"), mix2)
    np.testing.assert_array_equal(vb, vf)
    diff = np.abs(ob.astype(np.int32) - tensors.f32_to_bf16_bits(of).astype(np.int32))
    assert diff.max() <= 1
