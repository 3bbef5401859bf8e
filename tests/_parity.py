"""Shared helpers of the parity tests: run one outer step on the HIP engine
and on the CPU oracle from the same seeded inputs and compare them.

Tolerances (bars the engine must meet against the oracle):
  float32 outputs   over the whole output, max |gpu - ref| / max |ref| <= 1e-6; and
                    per worker row, max_p |gpu - ref| <= 1e-6 * max_p |ref| + delta,
                    where float32 rounding, which is relative to the operands, can
                    exceed 1e-6 of a row that cancels below them (one parameter per
                    worker: theta' = x - lr * step nearly 0 while x and lr * step are
                    not): delta = 32 * eps32 * max|theta_prev| for theta' (as for
                    bf16 below) and 32 * eps32 * max|v'| for v'
  bf16 theta'       at most 1 ulp apart (ordered-integer distance of the encodings),
                    or |gpu - ref| <= ulp(ref) + delta where the float32 evaluation
                    error itself exceeds half an ulp of the result
The float32 evaluation error of theta' is relative to the operands (the
mixed parameters, the mixed gradient), not to theta': where theta' nearly
cancels to 0 its bf16 ulp is tiny.  delta = 32 * eps32 * max|theta_prev|
bounds that error for up to 3 rounds of degree <= 4 (a few float32 roundings
per round, each relative to max|theta|); for a typical element delta is
~1/600 of an ulp, so those elements are held to 1 ulp.
  consensus rows    per row, max_m |gpu - ref| <= 1e-5 * max_m |ref| + floor; the
                    row of the stored theta' within a bound derived from the
                    element bar (theta_row_bound)
The consensus bound follows from float32 deviations: each deviation carries a
relative error of about eps32 * (2 |u| / |u - mean| + 2), at most ~1e-6 for
these inputs, doubled by squaring; 1e-5 leaves a factor of five.  The float32
mean of equal values need not equal them, so a row that is exactly 0 in
double precision can come out at the rounding floor
P * (4 * eps32 * max|theta|)^2, which is added as an absolute term.
"""

from __future__ import annotations

import numpy as np

import oracle
from synth import configs, graphs, tensors

F32_RTOL = 1e-6
CD_RTOL = 1e-5
EPS32 = 2.0 ** -24


def ordered_bf16(bits):
    """bf16 bit patterns -> integers ordered like the values they encode."""
    b = np.asarray(bits, dtype=np.int64)
    return np.where(b & 0x8000, 0x8000 - (b & 0x7FFF), 0x8000 + b)


def max_row_rel_err(got, ref):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    den = np.maximum(np.abs(ref).max(axis=1), 1e-300)
    return float((np.abs(got - ref).max(axis=1) / den).max()) if got.size else 0.0


def bf16_value(bits):
    return (np.asarray(bits, np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def bf16_ulp(bits):
    """Distance from |value| to the next bf16 value up in magnitude."""
    mag = np.asarray(bits, np.uint16) & 0x7FFF
    return bf16_value(mag + 1) - bf16_value(mag)


def _same_nonfinite(got, ref, what):
    """NaN exactly where the reference has NaN, the same infinities where it
    has infinities; returns the mask of elements finite on both sides."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    gn, rn = np.isnan(got), np.isnan(ref)
    assert np.array_equal(gn, rn), (f"{what}: NaN at {int((gn & ~rn).sum())} elements the reference has finite or "
                                    f"infinite, missing at {int((rn & ~gn).sum())}")
    gi, ri = np.isinf(got), np.isinf(ref)
    assert np.array_equal(gi, ri) and np.array_equal(got[ri], ref[ri]), f"{what}: infinities differ"
    return np.isfinite(ref)


def _check_f32(got, ref, delta, what):
    """Non-finite values where the reference has them; on the finite elements
    the whole-output relative bar and the per-row bar with the floor delta."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    if not got.size:
        return
    fin = _same_nonfinite(got, ref, what)
    g, r = np.where(fin, got, 0.0), np.where(fin, ref, 0.0)
    err = np.abs(g - r)
    e_all = float(err.max() / max(np.abs(r).max(), 1e-300))
    assert e_all <= F32_RTOL, f"{what} relative error {e_all:.3e} over the output"
    row_tol = F32_RTOL * np.abs(r).max(axis=1) + delta
    bad = err.max(axis=1) > row_tol
    assert not bad.any(), (f"{what}: rows {np.nonzero(bad)[0][:5].tolist()} exceed their bar "
                           f"(relative error {max_row_rel_err(g[bad], r[bad]):.3e}, floor {delta:.3e})")


def bf16_is_nan(bits):
    b = np.asarray(bits, np.uint16)
    return ((b & 0x7F80) == 0x7F80) & ((b & 0x007F) != 0)


def compare_outputs(dtype, got_t, ref_t, got_v, ref_v, P, theta_scale=None):
    """Asserts theta' and v' parity on [:, :P]; theta_scale = max|theta_prev|
    over its finite elements (needed for bf16; for float32 it sets the
    per-row floor, 0 without it).  Both outputs have NaN and infinities
    exactly where the oracle's have them; the bars hold on the rest."""
    got_v, ref_v = got_v[:, :P], ref_v[:, :P]
    fin_v = np.isfinite(np.asarray(ref_v, np.float64))
    v_scale = float(np.abs(np.asarray(ref_v, np.float64)[fin_v]).max()) if fin_v.any() else 0.0
    _check_f32(got_v, ref_v, 32 * EPS32 * v_scale if theta_scale is not None else 0.0, "momentum")
    if dtype == "f32":
        _check_f32(got_t[:, :P], ref_t[:, :P], 32 * EPS32 * theta_scale if theta_scale is not None else 0.0, "theta")
    else:
        g, r = got_t[:, :P], ref_t[:, :P]
        gn, rn = bf16_is_nan(g), bf16_is_nan(r)
        assert np.array_equal(gn, rn), f"theta: NaN at {int((gn ^ rn).sum())} elements the oracle does not match"
        g, r = np.where(rn, 0, g).astype(np.uint16), np.where(rn, 0, r).astype(np.uint16)
        ri = (r & 0x7FFF) == 0x7F80
        assert np.array_equal(g[ri], r[ri]), "theta: infinities differ"
        g, r = np.where(ri, 0, g).astype(np.uint16), np.where(ri, 0, r).astype(np.uint16)
        d = np.abs(ordered_bf16(g) - ordered_bf16(r))
        delta = 32 * EPS32 * theta_scale
        near_zero = np.abs(bf16_value(g) - bf16_value(r)) <= bf16_ulp(r) + delta
        bad = (d > 1) & ~near_zero
        assert not bad.any(), (f"theta differs by {d[bad].max()} bf16 ulps at {int(bad.sum())} elements "
                               f"(largest |ref| there {np.abs(bf16_value(r[bad])).max():.3e})")


def cd_floor(P, scale):
    """Absolute rounding floor of a float32-deviation sum over P parameters
    whose values are at most `scale` in magnitude: the float32 mean of equal
    values need not equal them, and a float32 square below the smallest
    subnormal 2^-149 rounds to a multiple of it (to 0 for deviations under
    2^-75), an absolute error of at most 2^-150 per term."""
    return P * (4 * EPS32 * scale) ** 2 + P * 2.0 ** -149


def compare_cd(got, ref, floor=0.0):
    """Per row, NaN where the oracle has NaN (a non-finite value in a row's
    input makes its worker mean, and so every S_m of the row, NaN) and
    max_m |gpu - ref| <= CD_RTOL * max_m |ref| + floor on the rest."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    assert got.shape == ref.shape
    for r in range(ref.shape[0]):
        fin = _same_nonfinite(got[r], ref[r], f"consensus row {r}")
        if not fin.any():
            continue
        tol = CD_RTOL * np.abs(ref[r][fin]).max() + floor
        err = np.abs(got[r][fin] - ref[r][fin]).max()
        assert err <= tol, f"consensus row {r}: error {err:.3e} > {tol:.3e} (ref max {np.abs(ref[r]).max():.3e})"


def topo(spec, M, rounds, seed=0, step=0):
    """Topology dict for a spec (see synth.configs.topology) plus test-only specs."""
    name = spec[0]
    if name == "matching":
        rp, ci, masks = graphs.random_matching_masks(M, rounds, seed)
        return dict(kind="csr", row_ptr=rp, col_idx=ci, weights=None, rounds=rounds, masks=masks,
                    reweight="metropolis")
    if name == "ring_self":
        rp, ci, w = graphs.ring_weights(M)
        masks = graphs.edge_drop_masks(rp, ci, rounds, spec[1], seed)
        return dict(kind="csr", row_ptr=rp, col_idx=ci, weights=w, rounds=rounds, masks=masks, reweight="self")
    if name == "er_mh":
        rp, ci = graphs.random_symmetric_structure(M, spec[1], seed)
        masks = graphs.edge_drop_masks(rp, ci, rounds, spec[2], seed + 1)
        return dict(kind="csr", row_ptr=rp, col_idx=ci, weights=None, rounds=rounds, masks=masks,
                    reweight="metropolis")
    if name == "complete":
        rp, ci, w = graphs.complete_weights(M)
        return dict(kind="csr", row_ptr=rp, col_idx=ci, weights=w, rounds=rounds, masks=None, reweight="none")
    return configs.topology(spec, M, rounds, seed, step)


last_variant = None  # the step kernel the last run_engine call launched (Engine.step_variant)


def run_engine(fgd, torch, M, P, ld, dtype, t1, t2, tp, tl, v, with_cd=True, lr=0.7, mu=0.9, nesterov=True,
               mix1_state=False, subset=None):
    """One step on the GPU.  Inputs are numpy arrays; returns numpy copies of
    (theta', v', cd or None)."""
    dev = torch.device("cuda:0")
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    if dtype == "f32":
        g_tp = torch.from_numpy(tp).to(dev)
        g_tl = torch.from_numpy(tl).to(dev)
    else:
        g_tp = torch.from_numpy(tp.view(np.int16)).to(dev).view(tdt)
        g_tl = torch.from_numpy(tl.view(np.int16)).to(dev).view(tdt)
    g_v = torch.from_numpy(v).to(dev)
    eng = fgd.Engine(M, P, ld, dtype, lr, mu, device=0, nesterov=nesterov, mix1_state=mix1_state)
    try:
        eng.set_topology_dict("mix1", t1)
        eng.set_topology_dict("mix2", t2)
        if subset is not None:
            eng.set_mix2_subset(subset)
        cd = None
        if with_cd:
            cd = torch.full((eng.num_cd_rows(), M), float("nan"), dtype=torch.float64, device=dev)
        global last_variant
        last_variant = eng.step_variant()
        eng.outer_step(g_tp, g_tl, g_v, cd)
        torch.cuda.synchronize()
    finally:
        eng.close()
    out_t = g_tp.cpu()
    out_t = out_t.numpy() if dtype == "f32" else out_t.view(torch.int16).numpy().view(np.uint16)
    return out_t, g_v.cpu().numpy(), (cd.cpu().numpy() if cd is not None else None)


def aligned_ld(P):
    """Smallest row stride >= P that keeps float32 and bf16 rows 16-byte aligned."""
    return max(8, -(-P // 8) * 8)


def run_case(fgd, torch, M, P, dtype, spec1, k1, spec2, k2, ld=None, seed=0, mom_std=1e-4, with_cd=True,
             lr=0.7, mu=0.9, nesterov=True, mix1_state=False, subset=None):
    ld = aligned_ld(P) if ld is None else ld
    tp, tl, v = tensors.numpy_inputs(M, P, ld=ld, dtype=dtype, mom_std=mom_std, seed=seed)
    t1 = topo(spec1, M, k1, seed)
    t2 = topo(spec2, M, k2, seed + 7)
    ref_t, ref_v, ref_cd = oracle.outer_step(tp, tl, v, oracle.Mix.from_topology(t1),
                                             oracle.Mix.from_topology(t2), lr=lr, mu=mu, P=P, dtype=dtype,
                                             nesterov=nesterov, mix1_state=mix1_state, subset=subset)
    got_t, got_v, got_cd = run_engine(fgd, torch, M, P, ld, dtype, t1, t2, tp, tl, v, with_cd, lr, mu,
                                      nesterov=nesterov, mix1_state=mix1_state, subset=subset)
    scale = float(np.abs(tensors.bf16_bits_to_f32(tp) if dtype == "bf16" else tp).max()) if tp.size else 0.0
    compare_outputs(dtype, got_t, ref_t, got_v, ref_v, P, scale)
    # The padding beyond P is never written.
    if ld > P:
        assert np.array_equal(got_t[:, P:], tp[:, P:]) and np.array_equal(got_v[:, P:], v[:, P:])
    if with_cd:
        compare_step_cd(got_cd, ref_cd, ref_t, dtype, P, scale)
    return got_t, got_v, got_cd


def theta_row_bound(ref_t, dtype, P, theta_scale):
    """Per-worker bound on |S_m(theta' as the engine stored it) - S_m(theta' as
    the oracle stored it)|, from the oracle's output alone.  Element (m, p) of
    the engine's theta' is within e[m, p] of the oracle's (the element bar
    compare_outputs enforces, plus float32 rounding of the deviation), the
    worker mean within max_n e[n, p]; with d the oracle's deviation, each term
    of the sum moves by at most 2 |d| D + D^2, D = e[m, p] + max_n e[n, p]."""
    r = np.asarray(ref_t[:, :P])
    val = bf16_value(r) if dtype == "bf16" else r.astype(np.float64)
    if dtype == "bf16":
        e = bf16_ulp(r) + 32 * EPS32 * theta_scale
    else:  # the float32 element bar: the whole-output bar and the row bar with its floor
        delta = 32 * EPS32 * theta_scale if theta_scale is not None else 0.0
        row = F32_RTOL * np.abs(val).max(axis=1, keepdims=True) + delta
        e = np.repeat(np.minimum(row, F32_RTOL * np.abs(val).max()), val.shape[1], axis=1)
    e = e + 4 * EPS32 * np.abs(val)
    D = e + e.max(axis=0, keepdims=True)
    d = val - val.mean(axis=0, keepdims=True)
    return (2 * np.abs(d) * D + D * D).sum(axis=1)


def compare_step_cd(got_cd, ref_cd, ref_t, dtype, P, theta_scale):
    """Every consensus row but the last against the oracle's (compare_cd); the
    last, S_m of the stored theta', within theta_row_bound of the oracle's."""
    got_cd = np.asarray(got_cd, np.float64)
    ref_cd = np.asarray(ref_cd, np.float64)
    compare_cd(got_cd[:-1], ref_cd[:-1], cd_floor(P, theta_scale))
    if not _same_nonfinite(got_cd[-1], ref_cd[-1], "theta' consensus row").all():
        return  # a non-finite theta' makes the row's worker mean, so every S_m, NaN
    bound = theta_row_bound(ref_t, dtype, P, theta_scale) + cd_floor(P, theta_scale)
    err = np.abs(got_cd[-1] - ref_cd[-1])
    assert np.all(err <= bound), f"theta' consensus row: error {err.max():.3e}, bound {bound[np.argmax(err - bound)]:.3e}"