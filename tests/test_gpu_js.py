"""GPU parity of the Jensen--Shannon functional distance (Sec. 4.4;
Appendix D.2) against the float64 oracle, through the C ABI.

The selected token sets are integer results and must match exactly (both
sides compare the stored logits, ties to the lower index).  The distances
are float64 on both sides with different summation orders and exp/log
implementations.  They are compared as JS = d^2 ln 2, the quantity both
sides sum: d = sqrt(JS / ln 2) would magnify the rounding of a JS near 0
(nearly identical workers) without bound.  Per token, each term
p (log p - log mix) has log-probabilities of magnitude at most
|z| + |lse| <= 2 max|z| + ln K, each carrying a few ulps of rounding, and the
probabilities over the selected tokens sum to at most 2, so two evaluations
differ by at most about 32 eps (max|z| + ln K + 1) plus the summation error
k eps JS; the bar is 4 times that.
"""

import numpy as np
import pytest

from oracle import js as ojs
from synth import logits as slog
from synth import tensors

pytestmark = pytest.mark.gpu

EPS = 2.0 ** -52
LN2 = float(np.log(2.0))


def _js_bar(zw, za, K, k, rd):
    """Bound on |JS_gpu - JS_ref| per entry of rd (see the module notes);
    max|z| is taken over the whole input, which only loosens it per token."""
    def fmax(a):
        a = np.asarray(a, np.float64)
        f = a[np.isfinite(a)]
        return float(np.abs(f).max()) if f.size else 0.0

    zmax = max(fmax(zw), fmax(za))
    return 128 * EPS * (zmax + np.log(K) + 1.0) + 4 * k * EPS * rd * rd * LN2


def _assert_d_close(d, rd, bar):
    """|d^2 - rd^2| ln 2 <= bar per entry; returns the implied bound on |d - rd|."""
    err = np.abs(d * d - rd * rd) * LN2
    assert np.all(err <= bar), f"JS differs by {err.max():.3e} (bar {np.min(bar):.3e})"
    return np.minimum(np.sqrt(bar / LN2), bar / (LN2 * np.maximum(d + rd, 1e-300)))


@pytest.fixture(scope="module")
def env():
    import torch

    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    import paper_2606_22768_amd as fgd

    return fgd, torch


def _values(a, dtype):
    return tensors.bf16_bits_to_f32(a) if dtype == "bf16" else a


def _workspace(fgd, torch, dtype, M, U):
    """The call's workspace, filled with a byte pattern: the kernels must
    not depend on what it held before."""
    return torch.full((fgd.fgd_js_workspace_size(dtype, M, U),), 0xA5, dtype=torch.uint8, device="cuda")


def _run(fgd, torch, A, W, dtype, K, k):
    U, ldk = A.shape
    M = W.shape[0]
    conv = (lambda x: torch.from_numpy(x.view(np.int16)).cuda().view(torch.bfloat16)) if dtype == "bf16" \
        else (lambda x: torch.from_numpy(x).cuda())
    gA, gW = conv(A), conv(W)
    d = torch.full((M, U), float("nan"), dtype=torch.float64, device="cuda")
    mean = torch.full((M,), float("nan"), dtype=torch.float64, device="cuda")
    tops = torch.full((U, k), -1, dtype=torch.int32, device="cuda")
    fgd.fgd_js_distance(gA, gW, dtype, M, U, K, ldk, k, d, mean, tops, _workspace(fgd, torch, dtype, M, U))
    torch.cuda.synchronize()
    return d.cpu().numpy(), mean.cpu().numpy(), tops.cpu().numpy()


def _check(fgd, torch, A, W, dtype, K, k):
    d, mean, tops = _run(fgd, torch, A, W, dtype, K, k)
    za = _values(A, dtype)[:, :K]
    zw = _values(W, dtype)[:, :, :K]
    rd, rmean, rtops = ojs.js_distances(zw, za, k)
    assert np.array_equal(tops, rtops), "top-k token sets differ"
    dbound = _assert_d_close(d, rd, _js_bar(zw, za, K, k, rd))
    assert np.all(np.abs(mean - rmean) <= dbound.mean(axis=1) + 1e-15)
    return d


CASES = [
    # (M, U, K, ldk, dtype, k)
    (8, 5, 1000, 1000, "f32", 100),
    (8, 5, 1000, 1008, "bf16", 100),
    (3, 7, 5003, 5008, "f32", 100),          # ragged vocabulary
    (3, 7, 5003, 5008, "bf16", 37),
    (1, 4, 32000, 32000, "bf16", 100),       # bf16: many exact ties among the logits
    (2, 3, 7, 8, "f32", 7),                  # full vocabulary (k = K)
    (2, 3, 500, 504, "bf16", 500),
    (2, 4, 2000, 2000, "f32", 257),          # k past the smaller per-token wave kernel
    (3, 5, 9000, 9008, "bf16", 400),
    (2, 4, 6000, 6000, "f32", 512),          # the wave kernel's largest k
    (2, 3, 4000, 4000, "bf16", 513),         # every token to the radix kernel
    (4, 2, 20000, 20000, "f32", 1024),       # largest k
    (5, 3, 3000, 3000, "bf16", 1),
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: f"M{c[0]}-U{c[1]}-K{c[2]}-{c[4]}-k{c[5]}")
def test_js_parity(env, case):
    fgd, torch = env
    M, U, K, ldk, dtype, k = case
    print(f"[js] {case}", flush=True)
    A, W = slog.numpy_logits(M, U, K, ldk, dtype, seed=K + M)
    _check(fgd, torch, A, W, dtype, K, k)


def test_js_ties_across_the_threshold(env):
    """Logits on a coarse grid: the k-th largest value is shared by many
    tokens, so the selection must split a tie (lower indices first)."""
    fgd, torch = env
    M, U, K, k = 3, 6, 4000, 100
    rng = np.random.default_rng(71)
    za = np.round(rng.standard_normal((U, K)) * 2).astype(np.float32)  # integers: huge ties
    zw = (za[None] + rng.standard_normal((M, U, K)).astype(np.float32) * np.float32(0.3)).astype(np.float32)
    _check(fgd, torch, za, zw, "f32", K, k)
    zb = np.zeros((U, K), np.float32)  # all equal: the first k tokens
    d, _, tops = _run(fgd, torch, zb, np.zeros((M, U, K), np.float32), "f32", K, k)
    assert np.array_equal(tops, np.tile(np.arange(k, dtype=np.int32), (U, 1)))
    assert np.all(d == 0.0)


def test_js_masked_tokens_and_signed_zero(env):
    """-inf logits (masked tokens) take no probability; -0 and +0 compare
    equal in the selection."""
    fgd, torch = env
    M, U, K, k = 2, 4, 2000, 100
    A, W = slog.numpy_logits(M, U, K, K, "f32", seed=5)
    A[:, ::3] = -np.inf
    W[:, :, ::5] = -np.inf
    A[:, 7], A[:, 8] = -0.0, 0.0
    _check(fgd, torch, A, W, "f32", K, k)


@pytest.mark.parametrize("noise", [1e-4, 1e-6, 1e-7])
def test_js_nearly_identical_workers(env, noise):
    """Workers whose float32 logits differ from the averaged model's by a
    few ulps or less: d from about 1e-5 down to about 1e-8, where the square
    root magnifies rounding most."""
    fgd, torch = env
    M, U, K, k = 4, 6, 5000, 100
    rng = np.random.default_rng(83)
    za = (rng.standard_normal((U, K)) * 2).astype(np.float32)
    zw = (za[None] + rng.standard_normal((M, U, K)) * noise).astype(np.float32)
    d = _check(fgd, torch, za, zw, "f32", K, k)
    assert np.all(d < 1e-3)


def test_js_identical_workers_are_zero(env):
    fgd, torch = env
    A, W = slog.numpy_logits(4, 3, 3000, 3000, "bf16", seed=9, noise=0.0)
    d, mean, _ = _run(fgd, torch, A, W, "bf16", 3000, 100)
    assert np.all(d == 0.0) and np.all(mean == 0.0)


def test_js_rejections(env):
    fgd, torch = env
    A = torch.zeros((2, 64), device="cuda")
    W = torch.zeros((3, 2, 64), device="cuda")
    d = torch.zeros((3, 2), dtype=torch.float64, device="cuda")
    need = fgd.fgd_js_workspace_size("f32", 3, 2)
    ws = torch.zeros(need + 64, dtype=torch.uint8, device="cuda")
    for kw in (dict(top_k=0), dict(top_k=65), dict(top_k=2000), dict(ldk=62, vocab=60), dict(vocab=65),
               dict(num_tokens=0), dict(dtype=7), dict(num_workers=0), dict(workspace=None),
               dict(workspace_bytes=need - 1), dict(workspace=ws[8:]), dict(workspace=d)):
        args = dict(dtype="f32", num_workers=3, num_tokens=2, vocab=64, ldk=64, top_k=10, workspace=ws,
                    workspace_bytes=None)
        args.update(kw)
        with pytest.raises(fgd.FgdError) as e:
            fgd.fgd_js_distance(A, W, args["dtype"], args["num_workers"], args["num_tokens"], args["vocab"],
                                args["ldk"], args["top_k"], d, workspace=args["workspace"],
                                workspace_bytes=args["workspace_bytes"] if args["workspace"] is not d else need)
        assert e.value.status == fgd.FGD_ERR_INVALID_ARG
    for bad in (dict(dtype=7), dict(num_workers=0), dict(num_tokens=0)):
        args = dict(dtype="f32", num_workers=3, num_tokens=2)
        args.update(bad)
        with pytest.raises(fgd.FgdError):
            fgd.fgd_js_workspace_size(args["dtype"], args["num_workers"], args["num_tokens"])


def test_js_full_size_sampled_tokens(env):
    """The benchmark's size (8 workers, 2048 tokens, 128256-token vocabulary,
    bf16): the distances and top-k sets of sampled tokens against the oracle
    (every token is independent, so the oracle on the sampled rows is exact
    parity for them), plus the mean over all tokens against the engine's own
    per-token distances summed in float64."""
    fgd, torch = env
    M, U, K, k = 8, 2048, 128256, 100
    print("[js] full size: generating logits", flush=True)
    A, W = slog.torch_logits(M, U, K, K, "bf16", seed=0)
    d = torch.empty((M, U), dtype=torch.float64, device="cuda")
    mean = torch.empty(M, dtype=torch.float64, device="cuda")
    tops = torch.empty((U, k), dtype=torch.int32, device="cuda")
    fgd.fgd_js_distance(A, W, "bf16", M, U, K, K, k, d, mean, tops, _workspace(fgd, torch, "bf16", M, U))
    torch.cuda.synchronize()
    rng = np.random.default_rng(0)
    sample = np.unique(np.concatenate([[0, U - 1], rng.integers(0, U, 14)]))
    za = A[sample].float().cpu().numpy()
    zw = W[:, sample].float().cpu().numpy()
    rd, _, rtops = ojs.js_distances(zw, za, k)
    assert np.array_equal(tops.cpu().numpy()[sample], rtops)
    _assert_d_close(d.cpu().numpy()[:, sample], rd, _js_bar(zw, za, K, k, rd))
    dh = d.cpu().numpy()
    np.testing.assert_allclose(mean.cpu().numpy(), dh.mean(axis=1), rtol=1e-13)
    assert np.all((dh > 0) & (dh < 1))
    print(f"[js] full size: CD_JS = {dh.mean():.6f}", flush=True)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_js_wide_logit_range(env, dtype):
    """Logits spread over hundreds of units: later values exceed a lane's
    running shift by more than the exponent slack (the rescale path), and
    most terms fall into the underflow range of exp."""
    fgd, torch = env
    M, U, K, k = 3, 4, 20000, 100
    A, W = slog.numpy_logits(M, U, K, K, "f32", seed=23, scale=60.0, head_boost=200.0)
    ramp = np.linspace(-900.0, 900.0, K, dtype=np.float32)
    A[1] += ramp                          # rising: the shift moves at almost every vector
    W[:, 1] += ramp
    A[2] -= ramp                          # falling: the first vector holds the maximum
    W[:, 2] -= ramp
    if dtype == "bf16":
        import torch as _t

        A = _t.from_numpy(A).to(_t.bfloat16).view(_t.int16).numpy().view(np.uint16)
        W = _t.from_numpy(W).to(_t.bfloat16).view(_t.int16).numpy().view(np.uint16)
    _check(fgd, torch, A, W, dtype, K, k)


# bf16 bit patterns on both sides of the worker-row kernel's exp table
# (2^-16 <= |v| < 64): inside, just outside, zeros, the smallest subnormal
# and -inf.
BF16_TABLE_EDGES = [0x3780, 0x377F, 0x427F, 0x4280, 0xB780, 0xB77F, 0xC27F, 0xC280,
                    0x0000, 0x8000, 0x0001, 0x8001, 0xFF80]


def test_js_bf16_table_edges_single_lanes(env):
    """Rows of ordinary bf16 logits (table terms) with one value from
    BF16_TABLE_EDGES at a different position in each row: that value's
    vector, and only it, takes the general path for the whole wave, and the
    two partial sums are merged.  15 rows: the last row pair of the
    two-row blocks is half empty."""
    fgd, torch = env
    M, U, K, k = 3, 5, 3001, 100
    A, W = slog.numpy_logits(M, U, K, K + 7, "bf16", seed=31)
    for m in range(M):
        for u in range(U):
            r = m * U + u
            W[m, u, (r * 613) % K] = BF16_TABLE_EDGES[r % len(BF16_TABLE_EDGES)]
    _check(fgd, torch, A, W, "bf16", K, k)


def test_js_bf16_table_edges_dense(env):
    """Every edge pattern many times in every row (most vectors of the rows
    take the general path), logits of magnitude beyond the table on whole
    rows (only the general path), and rows within it (only the table)."""
    fgd, torch = env
    M, U, K, k = 4, 6, 2500, 100
    A, W = slog.numpy_logits(M, U, K, K + 4, "bf16", seed=37)
    rng = np.random.default_rng(41)
    edges = np.array(BF16_TABLE_EDGES, np.uint16)
    for m in range(M):
        pos = rng.choice(K, 200, replace=False)
        W[m, 0, pos] = edges[rng.integers(0, edges.size, 200)]
    big = (rng.standard_normal((M, K)) * 3 + 100).astype(np.float32)  # |v| >= 64: general path only
    import torch as _t

    W[:, 1, :K] = _t.from_numpy(big).to(_t.bfloat16).view(_t.int16).numpy().view(np.uint16)
    W[:, 2, : K // 2] = W[:, 1, : K // 2]  # half general, half table
    W[:, 3, ::2] = 0xFF80                  # every other token masked
    _check(fgd, torch, A, W, "bf16", K, k)


def test_js_bf16_rows_beyond_the_persistent_grid(env):
    """More rows than the bf16 row kernel's persistent grid streams at once
    (3 blocks of two rows per compute unit), so its thread groups take
    several rows in turn, averaged and worker rows alike."""
    fgd, torch = env
    M, U, K, k = 4, 520, 700, 50
    A, W = slog.numpy_logits(M, U, K, K + 4, "bf16", seed=43)
    W[1, 7, 3] = 0xFF80
    W[2, 519, 699] = 0x4280
    _check(fgd, torch, A, W, "bf16", K, k)


@pytest.mark.parametrize("dtype,K", [("f32", 140_003), ("bf16", 270_001)])
def test_js_long_vocabularies(env, dtype, K):
    """Vocabularies of 140003 and 270001 logits: a row thread of the
    averaged row streams 137 (float32) or 132 (bf16) vectors and records
    four of them; a head of large logits placed at the row's end lies in
    its last vectors."""
    fgd, torch = env
    M, U, k = 2, 3, 100
    A, W = slog.numpy_logits(M, U, K, -(-K // 8) * 8, "f32", seed=K)  # 16-byte rows in both storages
    rng = np.random.default_rng(K)
    tail = rng.choice(np.arange(K - 20_000, K), 150, replace=False)
    A[:, tail] += 12.0
    W[:, :, tail] += 12.0
    if dtype == "bf16":
        import torch as _t

        A = _t.from_numpy(A).to(_t.bfloat16).view(_t.int16).numpy().view(np.uint16)
        W = _t.from_numpy(W).to(_t.bfloat16).view(_t.int16).numpy().view(np.uint16)
    _check(fgd, torch, A, W, dtype, K, k)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_js_top_tokens_crowded_in_one_row_thread(env, dtype):
    """Most of a token's top logits in the vectors of one row thread (every
    one of its first 24 vectors holds one): its four recorded vector maxima
    all reach the threshold, so the candidate pass reads all of that
    thread's vectors; a second token crowds them into two threads' vectors,
    a third into one vector."""
    fgd, torch = env
    M, U, K, k = 2, 3, 60_000, 100
    A, W = slog.numpy_logits(M, U, K, K, "f32", seed=99)
    per = 8 if dtype == "bf16" else 4
    stride = 256 * per                                   # elements between a row thread's vectors
    pos0 = np.array([5 * per + v * stride + (v % per) for v in range(24)])
    pos1 = np.concatenate([pos0, pos0 + 37 * per])
    A[0, pos0] += 15.0
    A[1, pos1] += 15.0
    A[2, 7 * per: 8 * per] += 15.0
    W[:, 0, pos0] += 15.0
    if dtype == "bf16":
        import torch as _t

        A = _t.from_numpy(A).to(_t.bfloat16).view(_t.int16).numpy().view(np.uint16)
        W = _t.from_numpy(W).to(_t.bfloat16).view(_t.int16).numpy().view(np.uint16)
    _check(fgd, torch, A, W, dtype, K, k)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_js_row_padding_is_never_used(env, dtype):
    """Elements in [K, ldk) of every row are read with the vectors that
    straddle K but never enter a sum, a maximum or the selection: padding of
    NaN, +-inf and huge values gives the same distances and token sets as
    zero padding."""
    fgd, torch = env
    M, U, K, k = 3, 4, 1001, 100
    per = 8 if dtype == "bf16" else 4
    ldk = -(-K // per) * per + per  # a ragged last vector and one whole vector of padding
    A, W = slog.numpy_logits(M, U, K, ldk, dtype, seed=61)
    d0, m0, t0 = _run(fgd, torch, A, W, dtype, K, k)
    junk = np.array([0x7FC0, 0x7F80, 0xFF80, 0x7F7F, 0xFF7F], np.uint16) if dtype == "bf16" else \
        np.array([np.nan, np.inf, -np.inf, 3e38, -3e38], np.float32)
    pad = np.resize(junk, ldk - K)
    A[:, K:] = pad
    W[:, :, K:] = pad
    d1, m1, t1 = _run(fgd, torch, A, W, dtype, K, k)
    assert np.array_equal(t0, t1)
    assert np.array_equal(d0, d1) and np.array_equal(m0, m1)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("sweeps,extra", [(1, -1), (1, 0), (1, 1), (2, 0), (2, 5), (3, 1), (3, -7)])
def test_js_sweep_boundaries(env, dtype, sweeps, extra):
    """Vocabularies around whole sweeps of a row (256 row threads x one
    16-byte vector each): a row of one sweep, one element more or less, two
    and three sweeps, a ragged last vector; the last sweep is the only one
    some lanes lack or hold in part."""
    fgd, torch = env
    per = 8 if dtype == "bf16" else 4
    K = sweeps * 256 * per + extra
    k = min(100, K)
    ldk = -(-K // per) * per
    print(f"[js] sweeps {sweeps} extra {extra} {dtype} K {K}", flush=True)
    A, W = slog.numpy_logits(3, 5, K, ldk, dtype, seed=K)
    _check(fgd, torch, A, W, dtype, K, k)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_js_hundreds_of_candidates(env, dtype):
    """Averaged rows with a wide tie at the k-th value: 60 tokens above it
    and t tokens on it (t = 90 .. 450, scattered), the rest below.  The
    threshold from the recorded vector maxima is the tied value, so the
    per-token selection sorts 60 + t candidates (past two per lane for most
    tokens, up to 512, the limit of the kernel that takes k = 100) and must
    split the tie by index."""
    fgd, torch = env
    M, U, K, k = 2, 6, 40_000, 100
    A, W = slog.numpy_logits(M, U, K, K, "f32", seed=83)
    rng = np.random.default_rng(84)
    A = np.clip(A, -6.0, 1.5).astype(np.float32)
    for u, t in enumerate((90, 150, 250, 330, 400, 450)):
        pos = rng.choice(K, size=60 + t, replace=False)
        A[u, pos[:60]] = 5.0 + rng.integers(0, 4, size=60).astype(np.float32)
        A[u, pos[60:]] = 3.0
    if dtype == "bf16":
        import torch as _t

        A = _t.from_numpy(A).to(_t.bfloat16).view(_t.int16).numpy().view(np.uint16)
        W = _t.from_numpy(W).to(_t.bfloat16).view(_t.int16).numpy().view(np.uint16)
    _check(fgd, torch, A, W, dtype, K, k)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_js_hundreds_of_candidates_large_k(env, dtype):
    """k = 400 (the per-token wave kernel for 256 < k <= 512): 300 tokens
    above a tied value and t on it (t = 120 .. 760), so 420 .. 1060
    candidates: sorted at eight or sixteen per lane, and the last token,
    past the kernel's 1024, handed to the radix kernel."""
    fgd, torch = env
    M, U, K, k = 2, 6, 40_000, 400
    A, W = slog.numpy_logits(M, U, K, K, "f32", seed=85)
    rng = np.random.default_rng(86)
    A = np.clip(A, -6.0, 1.5).astype(np.float32)
    for u, t in enumerate((120, 200, 450, 600, 720, 760)):
        pos = rng.choice(K, size=300 + t, replace=False)
        A[u, pos[:300]] = 5.0 + rng.integers(0, 4, size=300).astype(np.float32)
        A[u, pos[300:]] = 3.0
    if dtype == "bf16":
        import torch as _t

        A = _t.from_numpy(A).to(_t.bfloat16).view(_t.int16).numpy().view(np.uint16)
        W = _t.from_numpy(W).to(_t.bfloat16).view(_t.int16).numpy().view(np.uint16)
    _check(fgd, torch, A, W, dtype, K, k)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("k,top,tied", [(256, 200, 312), (256, 200, 313), (400, 300, 724), (400, 300, 725)])
def test_js_candidate_capacity_boundaries(env, dtype, k, top, tied):
    """Exactly as many candidates as a per-token wave kernel holds, and one
    more: `top` tokens above a tied value and `tied` tokens on it, the rest
    below, so the threshold from the recorded vector maxima is the tied
    value and the candidates number top + tied: 512 and 513 for k = 256 (the
    kernel for k <= 256 holds 512), 1024 and 1025 for k = 400 (the one for
    256 < k <= 512 holds 1024); one past the capacity goes to the radix
    kernel.  The tie at the k-th value is split by index."""
    fgd, torch = env
    M, U, K = 2, 2, 40_000
    A, W = slog.numpy_logits(M, U, K, K, "f32", seed=91)
    rng = np.random.default_rng(92)
    A = np.clip(A, -6.0, 1.5).astype(np.float32)
    for u in range(U):
        pos = rng.choice(K, size=top + tied, replace=False)
        A[u, pos[:top]] = 5.0 + rng.integers(0, 4, size=top).astype(np.float32)
        A[u, pos[top:]] = 3.0
    if dtype == "bf16":
        import torch as _t

        A = _t.from_numpy(A).to(_t.bfloat16).view(_t.int16).numpy().view(np.uint16)
        W = _t.from_numpy(W).to(_t.bfloat16).view(_t.int16).numpy().view(np.uint16)
    _check(fgd, torch, A, W, dtype, K, k)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_js_candidate_overflow_mixed_with_ordinary_tokens(env, dtype):
    """Tokens whose averaged row is one repeated logit give every element as
    a candidate of the per-token wave selection (more than it holds); those
    tokens alone are handed to the radix kernel, in the same call as
    ordinary tokens that the wave kernel finishes, and the workspace's junk
    flags must not make either kernel take or skip the wrong token."""
    fgd, torch = env
    M, U, K, k = 3, 9, 3000, 100
    A, W = slog.numpy_logits(M, U, K, K, dtype, seed=77)
    for u in (1, 4, 8):
        A[u, :K] = A[u, 0]
    _check(fgd, torch, A, W, dtype, K, k)


@pytest.mark.parametrize("k", [50, 300, 600])
def test_js_many_tokens_with_flagged_ones(env, k):
    """3000 tokens: more than the radix kernel's blocks, so each block walks
    several tokens' flags (k = 50 and 300, the two per-token wave kernels;
    every 37th token's averaged row is one repeated logit and so flagged)
    or several tokens (k = 600: every token goes to the radix kernel)."""
    fgd, torch = env
    M, U, K, ldk = 2, 3000, 700, 704
    A, W = slog.numpy_logits(M, U, K, ldk, "bf16", seed=k)
    A[::37, :K] = A[::37, :1]
    _check(fgd, torch, A, W, "bf16", K, k)


def test_js_workspace_reused_across_shapes(env):
    """One workspace serves calls of different sizes in turn (bf16, then
    float32 over fewer tokens, then bf16 again): each call writes what it
    reads, so the results equal those of calls with fresh workspaces."""
    fgd, torch = env
    shapes = [(4, 9, 3001, 3008, "bf16", 100), (2, 5, 777, 780, "f32", 300), (3, 11, 1500, 1504, "bf16", 10)]
    need = max(fgd.fgd_js_workspace_size(dt, M, U) for M, U, _, _, dt, _ in shapes)
    ws = torch.full((need,), 0x5A, dtype=torch.uint8, device="cuda")
    for i, (M, U, K, ldk, dtype, k) in enumerate(shapes):
        A, W = slog.numpy_logits(M, U, K, ldk, dtype, seed=900 + i)
        d0, _, t0 = _run(fgd, torch, A, W, dtype, K, k)
        conv = (lambda x: torch.from_numpy(x.view(np.int16)).cuda().view(torch.bfloat16)) if dtype == "bf16" \
            else (lambda x: torch.from_numpy(x).cuda())
        d = torch.empty((M, U), dtype=torch.float64, device="cuda")
        tops = torch.empty((U, k), dtype=torch.int32, device="cuda")
        fgd.fgd_js_distance(conv(A), conv(W), dtype, M, U, K, ldk, k, d, None, tops, ws)
        torch.cuda.synchronize()
        assert np.array_equal(d.cpu().numpy(), d0) and np.array_equal(tops.cpu().numpy(), t0)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_js_pattern_reference_reads_only(env, dtype):
    """The row kernel's access pattern without arithmetic (the bench's
    streaming reference) leaves the logits bit-identical, and takes the same
    argument checks as the distance."""
    fgd, torch = env
    M, U, K = 3, 700, 1001
    ldk = -(-K // 8) * 8
    A, W = slog.numpy_logits(M, U, K, ldk, dtype, seed=88)
    conv = (lambda x: torch.from_numpy(x.view(np.int16)).cuda().view(torch.bfloat16)) if dtype == "bf16" \
        else (lambda x: torch.from_numpy(x).cuda())
    gA, gW = conv(A), conv(W)
    ws = _workspace(fgd, torch, dtype, M, U)
    fgd.fgd_stream_js_pattern(gA, gW, dtype, M, U, K, ldk, ws)
    torch.cuda.synchronize()
    raw = (lambda t: t.view(torch.int16).cpu().numpy().view(np.uint16)) if dtype == "bf16" \
        else (lambda t: t.cpu().numpy())
    assert np.array_equal(raw(gA).view(np.uint8), A.view(np.uint8))
    assert np.array_equal(raw(gW).view(np.uint8), W.view(np.uint8))
    for kw in (dict(workspace_bytes=ws.numel() - 1), dict(vocab=ldk + 1), dict(num_workers=0)):
        args = dict(num_workers=M, vocab=K, workspace_bytes=None)
        args.update(kw)
        with pytest.raises(fgd.FgdError) as e:
            fgd.fgd_stream_js_pattern(gA, gW, dtype, args["num_workers"], U, args["vocab"], ldk, ws,
                                      args["workspace_bytes"])
        assert e.value.status == fgd.FGD_ERR_INVALID_ARG


def _random_js_case(i):
    """Seeded random JS configuration: workers, tokens, vocabulary (tiny,
    mid, large), row stride, storage, k up to 1024, and a logit kind: plain,
    heavy ties (integers), wide range (the rescale path), masked tokens, or
    rows of equal logits (the radix-select fallback)."""
    rng = np.random.default_rng(777 + i)
    M = int(rng.integers(1, 7))
    U = int(rng.integers(1, 5))
    K = int(rng.choice([int(rng.integers(1, 64)), int(rng.integers(64, 3000)), int(rng.integers(3000, 9000))]))
    dtype = str(rng.choice(["f32", "bf16"]))
    per = 4 if dtype == "f32" else 8
    ldk = (K + int(rng.integers(0, 3)) * per + per - 1) // per * per
    k = int(min(K, rng.choice([1, int(rng.integers(1, 100)), 100, int(rng.integers(100, 1025))])))
    kind = int(rng.integers(0, 5))
    za = rng.standard_normal((U, ldk)) * float(rng.choice([0.5, 2.0, 8.0]))
    if kind == 1:
        za = np.round(za)
    if kind == 2:
        za = za * 50
    zw = za[None] + rng.standard_normal((M, U, ldk)) * float(rng.choice([1e-3, 0.1, 1.0]))
    if kind == 3:  # masked tokens; every distribution keeps a finite logit
        ma = rng.random(ldk) < 0.2
        mw = rng.random(ldk) < 0.2
        ma[0] = mw[0] = False
        za[:, ma] = -np.inf
        zw[:, :, mw] = -np.inf
    if kind == 4:
        za[:] = za[:, :1]
        zw[:] = zw[:, :, :1]
    za, zw = za.astype(np.float32), zw.astype(np.float32)
    if dtype == "bf16":
        import torch

        za = torch.from_numpy(za).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
        zw = torch.from_numpy(zw).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    return M, U, K, ldk, dtype, k, za, zw


@pytest.mark.parametrize("i", range(300))
def test_js_random_configurations(env, i):
    fgd, torch = env
    M, U, K, ldk, dtype, k, A, W = _random_js_case(i)
    print(f"[js] random case {i}: M={M} U={U} K={K} ldk={ldk} {dtype} k={k}", flush=True)
    _check(fgd, torch, A, W, dtype, K, k)
