"""Pins for the oracle's step variants, each against something other than the
oracle itself (torch's optimizer, scipy dense products, brute-force sums):

  - plain momentum (the optimizer with Nesterov off);
  - Mix1 also applied to the outer-optimizer state (Appendix B, GlobalM1S and
    GlobalM1SLocalM2 in the further-ablations table);
  - Mix2 restricted to a subset of parameter segments (Sec. 4.1 and Appendix
    C, the GlobalM1LocalM2-subset configuration; identity elsewhere).

Runs on the CPU only.
"""

import numpy as np
import pytest
import scipy.sparse
import torch

import oracle
from synth import graphs, tensors

LR, MU = np.float32(0.7), np.float32(0.9)


def dense_W(row_ptr, col_idx, w):
    M = len(row_ptr) - 1
    return scipy.sparse.csr_matrix((np.asarray(w, np.float64), col_idx, row_ptr), shape=(M, M)).toarray()


def torch_sgd(param, grad, buf, nesterov):
    """One torch.optim.SGD step (float64) with a preloaded momentum buffer."""
    p = torch.nn.Parameter(torch.from_numpy(np.array(param, np.float64)))
    opt = torch.optim.SGD([p], lr=float(LR), momentum=float(MU), nesterov=nesterov)
    p.grad = torch.from_numpy(np.array(grad, np.float64))
    opt.state[p]["momentum_buffer"] = torch.from_numpy(np.array(buf, np.float64)).clone()
    opt.step()
    return p.detach().numpy(), opt.state[p]["momentum_buffer"].numpy()


def close(got, want, ulps=2):
    np.testing.assert_allclose(got, want, rtol=0, atol=np.abs(want).max() * ulps * 2.0 ** -24 + 1e-30)


# ------------------------------------------------------------ plain momentum

@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_plain_momentum_m1_matches_torch_sgd(dtype):
    """M = 1, Nesterov off: torch's SGD with momentum (no Nesterov), gradient
    theta_prev - theta_local, buffer preloaded with v."""
    P = 3001
    tp, tl, v = tensors.numpy_inputs(1, P, dtype=dtype, mom_std=1e-4, seed=21)
    out_t, out_v, _ = oracle.outer_step(tp, tl, v, oracle.Mix("identity"), oracle.Mix("identity"), lr=LR, mu=MU,
                                        nesterov=False)
    f = tensors.bf16_bits_to_f32 if dtype == "bf16" else (lambda a: a)
    want_t, want_v = torch_sgd(f(tp[0]), f(tp[0]).astype(np.float64) - f(tl[0]), v[0], nesterov=False)
    close(out_v[0], want_v)
    if dtype == "bf16":
        want_bits = np.array([oracle.bf16_from_double(x) for x in want_t], dtype=np.uint16)
        # Double rounding aside (torch rounds nothing here), the stored value is
        # the nearest bf16 of the double result.
        assert np.array_equal(out_t[0], want_bits)
    else:
        close(out_t[0], want_t)


def test_plain_momentum_diloco_reduction():
    """Equal theta_prev and v everywhere, global Mix2, Nesterov off: every
    worker takes torch's momentum-SGD step on the mean outer gradient."""
    M, P = 6, 513
    rng = np.random.default_rng(4)
    base = (rng.standard_normal(P) * 0.02).astype(np.float32)
    tp = np.tile(base, (M, 1))
    tl = (tp + rng.standard_normal((M, P)).astype(np.float32) * np.float32(1e-3)).astype(np.float32)
    vb = (rng.standard_normal(P) * 1e-4).astype(np.float32)
    out_t, out_v, cd = oracle.outer_step(tp, tl, np.tile(vb, (M, 1)), oracle.Mix("global"), oracle.Mix("global"),
                                         lr=LR, mu=MU, nesterov=False)
    gbar = (tp.astype(np.float64) - tl.astype(np.float64)).mean(axis=0)
    want_t, want_v = torch_sgd(base, gbar, vb, nesterov=False)
    for m in range(M):
        close(out_t[m], want_t, ulps=4)
        close(out_v[m], want_v, ulps=4)
    assert np.all(cd[-1] == 0.0)


def test_plain_momentum_differs_from_nesterov_by_closed_form():
    """Both forms from the same inputs with a ring Mix2: x - lr (g + mu v')
    (Nesterov) and x - lr v' (plain), g and v' built from a dense scipy
    product; the momentum update itself is common to both forms."""
    M, P = 3, 400
    tp, tl, v = tensors.numpy_inputs(M, P, mom_std=1e-3, seed=8)
    m2 = oracle.Mix("csr", *graphs.ring_weights(M), rounds=1)
    tn, vn, _ = oracle.outer_step(tp, tl, v, oracle.Mix("identity"), m2, lr=LR, mu=MU, nesterov=True)
    tq, vq, _ = oracle.outer_step(tp, tl, v, oracle.Mix("identity"), m2, lr=LR, mu=MU, nesterov=False)
    assert np.array_equal(vn, vq)  # the momentum update does not depend on the form
    W = dense_W(*graphs.ring_weights(M))
    g = W @ (tp.astype(np.float64) - tl.astype(np.float64))
    vnew = float(MU) * v.astype(np.float64) + g
    close(tn, tp - float(LR) * (g + float(MU) * vnew), ulps=4)
    close(tq, tp - float(LR) * vnew, ulps=4)


# ------------------------------------------------------ Mix1 over the state

@pytest.mark.parametrize("nesterov", [True, False])
def test_global_state_mix_matches_torch_on_mean_buffer(nesterov):
    """GlobalM1S with ring Mix2 (GlobalM1SLocalM2): worker m's result is
    torch's SGD step from the worker-mean parameters with gradient (W2 g0)_m
    and the momentum buffer preloaded with the worker mean of v."""
    M, P = 8, 700
    tp, tl, v = tensors.numpy_inputs(M, P, mom_std=1e-3, seed=13)
    rp, ci, w = graphs.ring_weights(M)
    out_t, out_v, _ = oracle.outer_step(tp, tl, v, oracle.Mix("global"), oracle.Mix("csr", rp, ci, w, rounds=1),
                                        lr=LR, mu=MU, nesterov=nesterov, mix1_state=True)
    W2 = dense_W(rp, ci, w)
    g = W2 @ (tp.astype(np.float64) - tl.astype(np.float64))
    xbar = tp.astype(np.float64).mean(axis=0)
    vbar = v.astype(np.float64).mean(axis=0)
    for m in range(M):
        want_t, want_v = torch_sgd(xbar, g[m], vbar, nesterov)
        close(out_t[m], want_t, ulps=4)
        close(out_v[m], want_v, ulps=4)


def test_csr_state_mix_matches_dense_products():
    """Mix1 over a CSR W1 (two rounds, directed exponential graph) applied to
    both theta_prev and v: worker m steps from (W1^2 theta)_m with buffer
    (W1^2 v)_m, via torch's SGD."""
    M, P = 16, 300
    tp, tl, v = tensors.numpy_inputs(M, P, mom_std=1e-3, seed=17)
    rp, ci, w = graphs.exponential_weights(M)
    m1 = oracle.Mix("csr", rp, ci, w, rounds=2)
    out_t, out_v, _ = oracle.outer_step(tp, tl, v, m1, oracle.Mix("identity"), lr=LR, mu=MU, mix1_state=True)
    W1 = dense_W(rp, ci, w)
    x = W1 @ (W1 @ tp.astype(np.float64))
    vb = W1 @ (W1 @ v.astype(np.float64))
    g = tp.astype(np.float64) - tl.astype(np.float64)
    for m in range(M):
        want_t, want_v = torch_sgd(x[m], g[m], vb[m], True)
        close(out_t[m], want_t, ulps=4)
        close(out_v[m], want_v, ulps=4)


def test_state_mix_off_leaves_momentum_per_worker():
    """Without state mixing the new momentum is mu v_m + g_m per worker, with
    the same Mix1 (the state is not mixed unless asked)."""
    M, P = 4, 64
    tp, tl, v = tensors.numpy_inputs(M, P, mom_std=1e-3, seed=2)
    _, out_v, _ = oracle.outer_step(tp, tl, v, oracle.Mix("global"), oracle.Mix("identity"), lr=LR, mu=MU)
    close(out_v, float(MU) * v.astype(np.float64) + (tp.astype(np.float64) - tl.astype(np.float64)))


# -------------------------------------------------------------- Mix2 subset

SEGMENT_CASES = [
    [(0, 100)],
    [(37, 38), (200, 257), (511, 600)],
    [(0, 600)],
    [(599, 600)],
]


@pytest.mark.parametrize("segs", SEGMENT_CASES)
def test_subset_plain_sgd_factored_form(segs):
    """lr = 1, mu = 0: theta' = Mix1(theta) + Mix2_S(Delta), where Mix2_S is K2
    rounds of W2 on the subset columns and the identity elsewhere, built here
    as dense scipy products column by column."""
    M, P = 6, 600
    tp, tl, v = tensors.numpy_inputs(M, P, mom_std=0.0, seed=23)
    rp, ci, w = graphs.ring_weights(M)
    W = dense_W(rp, ci, w)
    out_t, _, cd = oracle.outer_step(tp, tl, np.zeros_like(v), oracle.Mix("global"),
                                     oracle.Mix("csr", rp, ci, w, rounds=2), lr=1.0, mu=0.0, subset=segs)
    inset = np.zeros(P, bool)
    for b, e in segs:
        inset[b:e] = True
    d = tl.astype(np.float64) - tp.astype(np.float64)
    dm = np.where(inset[None, :], W @ (W @ d), d)
    want = tp.astype(np.float64).mean(axis=0)[None, :] + dm
    close(out_t, want, ulps=4)
    # Consensus rows of the Mix2 rounds: brute-force sums over both parts.
    g0 = -d
    for k, gk in enumerate([g0, np.where(inset, W @ g0, g0), np.where(inset, W @ (W @ g0), g0)]):
        S = ((gk - gk.mean(axis=0)) ** 2).sum(axis=1)
        np.testing.assert_allclose(cd[k], S, rtol=1e-12, atol=1e-300)


def test_subset_segments_match_full_and_no_mix2():
    """Inside the subset the result equals the full-Mix2 step, outside it the
    step with Mix2 the identity (Nesterov, random momentum)."""
    M, P = 8, 1000
    tp, tl, v = tensors.numpy_inputs(M, P, dtype="bf16", mom_std=1e-3, seed=29)
    rp, ci, w = graphs.ring_weights(M)
    m2 = oracle.Mix("csr", rp, ci, w, rounds=1)
    segs = [(0, 129), (400, 401), (700, 1000)]
    ts, vs, _ = oracle.outer_step(tp, tl, v, oracle.Mix("global"), m2, subset=segs)
    tf, vf, _ = oracle.outer_step(tp, tl, v, oracle.Mix("global"), m2)
    tn, vn, _ = oracle.outer_step(tp, tl, v, oracle.Mix("global"), oracle.Mix("identity"))
    inset = np.zeros(P, bool)
    for b, e in segs:
        inset[b:e] = True
    assert np.array_equal(ts[:, inset], tf[:, inset]) and np.array_equal(vs[:, inset], vf[:, inset])
    assert np.array_equal(ts[:, ~inset], tn[:, ~inset]) and np.array_equal(vs[:, ~inset], vn[:, ~inset])


@pytest.mark.parametrize("segs", [[(5, 5)], [(10, 20), (15, 30)], [(30, 40), (10, 20)], [(0, 601)], [(-1, 3)]])
def test_subset_rejects_bad_segments(segs):
    M, P = 2, 600
    tp, tl, v = tensors.numpy_inputs(M, P, seed=1)
    with pytest.raises(ValueError):
        oracle.outer_step(tp, tl, v, oracle.Mix("global"), oracle.Mix("global"), subset=segs)


# ---------------------------------------------------------- split execution

def _store(a, dtype):
    """Rounded to the parameter storage type, back in float64 (torch's RNE casts)."""
    t = torch.from_numpy(np.asarray(a, np.float64))
    return (t.to(torch.bfloat16) if dtype == "bf16" else t.to(torch.float32)).to(torch.float64).numpy()


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("state", [False, True])
@pytest.mark.parametrize("nesterov", [True, False])
def test_split_halves_match_torch_from_stored_x(dtype, state, nesterov):
    """Algorithm 1 split: x = W1^2 theta stored in the parameter type, the
    state (optionally) replaced by W1^2 v in float32, then the blocking half
    from the stored x with ghat = W2 g0 on a subset: worker m's result is
    torch's SGD step from the stored x_m, gradient ghat_m, buffer v_m.
    Consensus rows against brute-force sums."""
    M, P = 8, 900
    tp, tl, v = tensors.numpy_inputs(M, P, dtype=dtype, mom_std=1e-3, seed=47)
    f = tensors.bf16_bits_to_f32 if dtype == "bf16" else (lambda a: a)
    rp1, ci1, w1 = graphs.exponential_weights(M, hops=(1, 2, 4))
    rp2, ci2, w2 = graphs.ring_weights(M)
    m1 = oracle.Mix("csr", rp1, ci1, w1, rounds=2)
    m2 = oracle.Mix("csr", rp2, ci2, w2, rounds=1)
    segs = [(0, 300), (600, 901 - 1)]
    x, v1, cd1 = oracle.mix1_split(tp, m1, mom=v, mix1_state=state)
    tq, tlq, vq, cd2 = oracle.outer_blocking(x, tp, tl, v1 if state else v, m2, lr=LR, mu=MU, nesterov=nesterov,
                                             subset=segs, write_local=True)

    W1, W2 = dense_W(rp1, ci1, w1), dense_W(rp2, ci2, w2)
    th = f(tp).astype(np.float64)
    xd = W1 @ (W1 @ th)
    np.testing.assert_array_equal(f(x).astype(np.float64), _store(xd, dtype))
    for k, u in enumerate([th, W1 @ th, xd]):
        np.testing.assert_allclose(cd1[k], ((u - u.mean(axis=0)) ** 2).sum(axis=1), rtol=1e-12)
    vb = _store(W1 @ (W1 @ v.astype(np.float64)), "f32") if state else v.astype(np.float64)
    if state:
        np.testing.assert_array_equal(v1.astype(np.float64), vb)
    g0 = th - f(tl).astype(np.float64)
    inset = np.zeros(P, bool)
    for b, e in segs:
        inset[b:e] = True
    gh = np.where(inset, W2 @ g0, g0)
    for m in range(M):
        want_t, want_v = torch_sgd(_store(xd[m], dtype), gh[m], vb[m], nesterov)
        close(vq[m], want_v, ulps=4)
        if dtype == "bf16":
            want_bits = np.array([oracle.bf16_from_double(t) for t in want_t], dtype=np.uint16)
            d = np.abs(want_bits.astype(np.int32) - tq[m].astype(np.int32))
            assert d.max() <= 1  # torch's double result may sit on the other side of a tie
        else:
            close(tq[m], want_t, ulps=4)
    assert np.array_equal(tlq, tq)  # theta' written back as the next inner start
    np.testing.assert_allclose(cd2[0], ((g0 - g0.mean(axis=0)) ** 2).sum(axis=1), rtol=1e-12)
    np.testing.assert_allclose(cd2[1], ((gh - gh.mean(axis=0)) ** 2).sum(axis=1), rtol=1e-12)
    ts = f(tq).astype(np.float64)
    np.testing.assert_allclose(cd2[2], ((ts - ts.mean(axis=0)) ** 2).sum(axis=1), rtol=1e-12)


def test_split_without_write_back_keeps_theta_local():
    M, P = 4, 128
    tp, tl, v = tensors.numpy_inputs(M, P, mom_std=1e-3, seed=3)
    x, _, _ = oracle.mix1_split(tp, oracle.Mix("global"))
    _, tlq, _, _ = oracle.outer_blocking(x, tp, tl, v, oracle.Mix("global"))
    assert np.array_equal(tlq, tl)
    # A global Mix1 stores the same x for every worker.
    assert np.all(x == x[0])


# --------------------------------------------------------------- JS distance

import scipy.spatial.distance  # noqa: E402

from oracle import js as ojs  # noqa: E402


def _logits(rng, K, scale=2.0):
    return rng.standard_normal(K) * scale


@pytest.mark.parametrize("K", [7, 100, 1000])
def test_js_full_vocabulary_matches_scipy(K):
    """k = K: the restricted sum is the full JS divergence, and d equals
    scipy's jensenshannon(p, q, base=2) of the two softmax distributions."""
    rng = np.random.default_rng(K)
    for _ in range(5):
        za = _logits(rng, K)
        zw = za + rng.standard_normal(K) * 0.3
        p = np.exp(zw - zw.max()); p /= p.sum()
        q = np.exp(za - za.max()); q /= q.sum()
        want = scipy.spatial.distance.jensenshannon(p, q, base=2)
        assert abs(ojs.js_distance_token(zw, za, K) - want) <= 1e-12


def test_js_identical_is_zero_and_disjoint_is_one():
    rng = np.random.default_rng(3)
    za = _logits(rng, 500)
    assert ojs.js_distance_token(za, za, 100) == 0.0
    assert ojs.js_distance_token(za + 3.0, za, 500) <= 1e-7  # logits shifted: same distribution
    # Distributions concentrated on different tokens: distance 1 (normalized maximum).
    a = np.full(50, -1e4); a[3] = 0.0
    b = np.full(50, -1e4); b[17] = 0.0
    assert abs(ojs.js_distance_token(a, b, 50) - 1.0) <= 1e-12


def test_js_masked_tokens_contribute_nothing():
    """A token of probability 0 on one side adds nothing to that side's KL
    term (0 log 0 = 0): masking tokens with -inf logits equals scipy's JS on
    distributions with those probabilities set to 0."""
    rng = np.random.default_rng(12)
    K = 300
    za, zw = _logits(rng, K), _logits(rng, K)
    za[::7] = -np.inf
    zw[::5] = -np.inf
    p = np.exp(zw - zw[np.isfinite(zw)].max()); p /= p.sum()
    q = np.exp(za - za[np.isfinite(za)].max()); q /= q.sum()
    want = scipy.spatial.distance.jensenshannon(p, q, base=2)
    assert abs(ojs.js_distance_token(zw, za, K) - want) <= 1e-12
    both = np.full(K, -np.inf); both[:3] = [0.0, 1.0, 2.0]
    assert ojs.js_distance_token(both, both, K) == 0.0


def test_js_restricted_sum_is_monotone_in_k():
    """Every term is non-negative: d grows with k and reaches the full value."""
    rng = np.random.default_rng(9)
    K = 800
    za = _logits(rng, K)
    zw = za + rng.standard_normal(K) * 0.5
    ds = [ojs.js_distance_token(zw, za, k) for k in (1, 10, 100, 400, K)]
    assert all(a <= b + 1e-15 for a, b in zip(ds, ds[1:]))
    p = np.exp(zw - zw.max()); p /= p.sum()
    q = np.exp(za - za.max()); q /= q.sum()
    assert abs(ds[-1] - scipy.spatial.distance.jensenshannon(p, q, base=2)) <= 1e-12


def test_js_top_k_by_brute_force_with_ties():
    """The top-k set against a brute-force selection by repeated argmax
    (first occurrence wins, so ties go to the lower index)."""
    rng = np.random.default_rng(5)
    z = np.round(rng.standard_normal(300) * 2, 1)  # many exact ties
    for k in (1, 5, 37, 100, 300):
        left = list(z)
        picked = []
        for _ in range(k):
            i = int(np.argmax(left))
            picked.append(i)
            left[i] = -np.inf
        assert np.array_equal(ojs.top_k_indices(z, k), np.sort(picked))


def test_js_distances_shapes_and_means():
    rng = np.random.default_rng(2)
    M, U, K = 3, 4, 64
    za = rng.standard_normal((U, K))
    zw = za[None] + rng.standard_normal((M, U, K)) * 0.2
    d, mean, tops = ojs.js_distances(zw, za, k=10)
    assert d.shape == (M, U) and mean.shape == (M,) and tops.shape == (U, 10)
    np.testing.assert_allclose(mean, d.mean(axis=1), rtol=0, atol=0)
    assert np.all((d > 0) & (d < 1))
