"""Seeded parameter, local-parameter and momentum tensors for the outer step.

Layout is worker-major ``[M][ld]`` with ``ld >= P``; only ``[:, :P]`` is
meaningful.  Recipe (per worker row, i.i.d. per element):

    theta_prev  ~ N(0, prev_std)
    theta_local = theta_prev + N(0, drift_std)
    momentum    ~ N(0, mom_std)        (exactly zero when mom_std == 0)

Values are drawn in float32.  For bf16 storage the float32 draws of
theta_prev and theta_local are rounded to bf16 (round to nearest even) by
torch's dtype conversion; momentum stays float32.

``numpy_inputs`` serves CPU-sized cases; ``torch_inputs`` generates on a
torch device with torch's counter-based generator, row by row, so that a
multi-gigabyte configuration never needs a host copy.
"""

from __future__ import annotations

import numpy as np


def numpy_inputs(M, P, ld=None, dtype="f32", prev_std=0.02, drift_std=1e-3, mom_std=1e-4, seed=0):
    """Returns (theta_prev, theta_local, momentum) as numpy arrays [M][ld].

    dtype "f32": float32 arrays.  dtype "bf16": uint16 arrays holding bf16 bit
    patterns for the two parameter tensors; momentum is float32.
    """
    ld = P if ld is None else ld
    if ld < P:
        raise ValueError("ld < P")
    rng = np.random.Generator(np.random.PCG64(seed))
    tp = np.zeros((M, ld), dtype=np.float32)
    tl = np.zeros((M, ld), dtype=np.float32)
    v = np.zeros((M, ld), dtype=np.float32)
    tp[:, :P] = rng.standard_normal((M, P), dtype=np.float32) * np.float32(prev_std)
    tl[:, :P] = tp[:, :P] + rng.standard_normal((M, P), dtype=np.float32) * np.float32(drift_std)
    if mom_std:
        v[:, :P] = rng.standard_normal((M, P), dtype=np.float32) * np.float32(mom_std)
    if dtype == "f32":
        return tp, tl, v
    if dtype == "bf16":
        return f32_to_bf16_bits(tp), f32_to_bf16_bits(tl), v
    raise ValueError(dtype)


def f32_to_bf16_bits(a):
    """float32 numpy array -> uint16 bf16 bit patterns (RNE via torch's conversion)."""
    import torch

    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16).copy()


def bf16_bits_to_f32(b):
    """uint16 bf16 bit patterns -> float32 (exact widening)."""
    b = np.ascontiguousarray(b, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32)


def torch_inputs(M, P, ld=None, dtype="f32", prev_std=0.02, drift_std=1e-3, mom_std=1e-4, seed=0,
                 device="cuda", out=None):
    """Returns (theta_prev, theta_local, momentum) torch tensors [M][ld] on device.

    Row m is drawn from a generator seeded with seed * 1_000_003 + m so that
    any row can be regenerated alone.  With ``out`` = (theta_prev,
    theta_local, momentum), [M][ld] tensors of the right dtypes allocated by
    the caller, those are filled (zeros outside [:, :P]) and returned.
    """
    import torch

    ld = P if ld is None else ld
    pdt = torch.float32 if dtype == "f32" else torch.bfloat16
    if out is None:
        tp = torch.zeros((M, ld), dtype=pdt, device=device)
        tl = torch.zeros((M, ld), dtype=pdt, device=device)
        v = torch.zeros((M, ld), dtype=torch.float32, device=device)
    else:
        tp, tl, v = out
        for t, dt in ((tp, pdt), (tl, pdt), (v, torch.float32)):
            if t.shape != (M, ld) or t.dtype != dt:
                raise ValueError(f"out tensor {tuple(t.shape)} {t.dtype}: expected ({M}, {ld}) {dt}")
            t.zero_()
        device = tp.device
    g = torch.Generator(device=device)
    for m in range(M):
        g.manual_seed(seed * 1_000_003 + m)
        a = torch.randn(P, generator=g, device=device, dtype=torch.float32).mul_(prev_std)
        b = torch.randn(P, generator=g, device=device, dtype=torch.float32).mul_(drift_std).add_(a)
        tp[m, :P] = a.to(pdt)
        tl[m, :P] = b.to(pdt)
        del a, b
        if mom_std:
            v[m, :P] = torch.randn(P, generator=g, device=device, dtype=torch.float32).mul_(mom_std)
    return tp, tl, v
