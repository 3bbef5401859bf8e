"""Python view of the CPU oracle (``fgd_oracle.c``).

TEST INFRASTRUCTURE.  Only the tests, ``__graft_entry__.smoke()`` and the
benchmark's CPU-baseline leg may import this package.  The product path (the
HIP engine and its binding) never imports it, and it never imports the
product.

The oracle follows the paper's outer step in double precision (Sec. 3 gossip
mixing operator and DiLoCo equations, Sec. 4.1 factored formulation,
Appendix A Algorithm 1, Appendix B Nesterov implementation form, Sec. 4.4 and
Appendix D.1 consensus distance).  Every function here is marshalling only.
"""

from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "fgd_oracle.c")
_LIB = os.path.join(_HERE, "libfgd_oracle.so")

KIND = {"identity": 0, "global": 1, "csr": 2}
REWEIGHT = {"none": 0, "metropolis": 1, "self": 2}


def build(force: bool = False) -> str:
    """Compile the oracle with gcc: -O2, no fast-math, no OpenMP, no SIMD flags."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fno-fast-math",
                               "-ffp-contract=off", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


class _Mix(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("rounds", ctypes.c_int32),
                ("row_ptr", ctypes.c_void_p), ("col_idx", ctypes.c_void_p),
                ("weights", ctypes.c_void_p), ("masks", ctypes.c_void_p),
                ("reweight", ctypes.c_int32)]


class _Opts(ctypes.Structure):
    _fields_ = [("lr", ctypes.c_float), ("mu", ctypes.c_float), ("nesterov", ctypes.c_int32),
                ("mix1_state", ctypes.c_int32), ("n_seg", ctypes.c_int32), ("seg", ctypes.c_void_p)]


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        L = ctypes.CDLL(_LIB)
        L.fgdo_bf16_from_double.restype = ctypes.c_uint16
        L.fgdo_bf16_from_double.argtypes = [ctypes.c_double]
        L.fgdo_round_weights.restype = ctypes.c_int
        L.fgdo_round_weights.argtypes = [ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                         ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p]
        L.fgdo_mix_apply.restype = ctypes.c_int
        L.fgdo_mix_apply.argtypes = [ctypes.c_int32, ctypes.c_int64, ctypes.POINTER(_Mix), ctypes.c_void_p,
                                     ctypes.c_void_p, ctypes.c_void_p]
        L.fgdo_num_cd.restype = ctypes.c_int
        L.fgdo_num_cd.argtypes = [ctypes.POINTER(_Mix), ctypes.POINTER(_Mix)]
        L.fgdo_outer_step.restype = ctypes.c_int
        L.fgdo_outer_step.argtypes = [ctypes.c_int32, ctypes.c_int64, ctypes.c_int64, ctypes.c_int32,
                                      ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                      ctypes.POINTER(_Mix), ctypes.POINTER(_Mix), ctypes.POINTER(_Opts),
                                      ctypes.c_void_p]
        L.fgdo_mix1_split.restype = ctypes.c_int
        L.fgdo_mix1_split.argtypes = [ctypes.c_int32, ctypes.c_int64, ctypes.c_int64, ctypes.c_int32,
                                      ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.POINTER(_Mix),
                                      ctypes.c_int32, ctypes.c_void_p]
        L.fgdo_outer_blocking.restype = ctypes.c_int
        L.fgdo_outer_blocking.argtypes = [ctypes.c_int32, ctypes.c_int64, ctypes.c_int64, ctypes.c_int32,
                                          ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                          ctypes.POINTER(_Mix), ctypes.POINTER(_Opts), ctypes.c_int32,
                                          ctypes.c_void_p]
        L.fgdo_consensus.restype = ctypes.c_int
        L.fgdo_consensus.argtypes = [ctypes.c_int32, ctypes.c_int64, ctypes.c_int64, ctypes.c_int32,
                                     ctypes.c_void_p, ctypes.c_void_p]
        _lib = L
    return _lib


def _ptr(a):
    return None if a is None else a.ctypes.data


class Mix:
    """One Mix slot as the oracle takes it.  Keeps its arrays alive."""

    def __init__(self, kind="identity", row_ptr=None, col_idx=None, weights=None, rounds=0, masks=None,
                 reweight="none"):
        self.kind = kind
        self.row_ptr = None if row_ptr is None else np.ascontiguousarray(row_ptr, dtype=np.int32)
        self.col_idx = None if col_idx is None else np.ascontiguousarray(col_idx, dtype=np.int32)
        self.weights = None if weights is None else np.ascontiguousarray(weights, dtype=np.float32)
        self.masks = None if masks is None else np.ascontiguousarray(masks, dtype=np.uint8)
        self.rounds = int(rounds)
        self.reweight = reweight

    @classmethod
    def from_topology(cls, t):
        """From the dict produced by synth.configs.topology."""
        return cls(kind=t["kind"], row_ptr=t["row_ptr"], col_idx=t["col_idx"], weights=t["weights"],
                   rounds=t["rounds"], masks=t["masks"], reweight=t["reweight"])

    def c(self):
        return _Mix(KIND[self.kind], self.rounds, _ptr(self.row_ptr), _ptr(self.col_idx), _ptr(self.weights),
                    _ptr(self.masks), REWEIGHT[self.reweight])

    def effective_rounds(self):
        return {"identity": 0, "global": 1}.get(self.kind, self.rounds)


def bf16_from_double(x: float) -> int:
    return int(lib().fgdo_bf16_from_double(float(x)))


def round_weights(row_ptr, col_idx, weights, mask, reweight):
    """Effective float32 weights of one round (raises on invalid input)."""
    row_ptr = np.ascontiguousarray(row_ptr, dtype=np.int32)
    col_idx = np.ascontiguousarray(col_idx, dtype=np.int32)
    w = None if weights is None else np.ascontiguousarray(weights, dtype=np.float32)
    mk = None if mask is None else np.ascontiguousarray(mask, dtype=np.uint8)
    out = np.zeros(col_idx.shape[0], dtype=np.float32)
    rc = lib().fgdo_round_weights(len(row_ptr) - 1, _ptr(row_ptr), _ptr(col_idx), _ptr(w), _ptr(mk),
                                  REWEIGHT[reweight], _ptr(out))
    if rc:
        raise ValueError(f"oracle rejected the topology (rc={rc})")
    return out


def mix_apply(mix: Mix, src):
    """All rounds of one Mix on a double [M][P] array.  Returns (dst, cd[(K+1), M])."""
    src = np.ascontiguousarray(src, dtype=np.float64)
    M, P = src.shape
    dst = np.empty_like(src)
    cd = np.zeros((mix.effective_rounds() + 1, M), dtype=np.float64)
    c = mix.c()
    rc = lib().fgdo_mix_apply(M, P, ctypes.byref(c), _ptr(src), _ptr(dst), _ptr(cd))
    if rc:
        raise ValueError(f"oracle mix failed (rc={rc})")
    return dst, cd


def num_cd(mix1: Mix, mix2: Mix) -> int:
    return mix2.effective_rounds() + 1 + mix1.effective_rounds() + 1 + 1


def subset_array(segments):
    """[n][2] int64 array of half-open Mix2 subset segments (None: no subset)."""
    if segments is None:
        return None
    return np.ascontiguousarray(np.asarray(segments, dtype=np.int64).reshape(-1, 2))


def outer_step(theta_prev, theta_local, mom, mix1: Mix, mix2: Mix, lr=0.7, mu=0.9, P=None, dtype=None,
               nesterov=True, mix1_state=False, subset=None):
    """One outer step.  Inputs are numpy [M][ld] arrays (float32, or uint16 bf16
    bits for the parameter tensors).  Returns new copies
    (theta_prev', mom', cd[n_cd, M]); the inputs are left untouched.

    nesterov: Nesterov (App. B two-line form) or plain momentum.
    mix1_state: Mix1 also mixes the momentum (App. B, GlobalM1S).
    subset: Mix2 acts only on these [begin, end) parameter segments."""
    tp = np.array(theta_prev, copy=True, order="C")
    tl = np.ascontiguousarray(theta_local)
    v = np.array(mom, dtype=np.float32, copy=True, order="C")
    if dtype is None:
        dtype = "bf16" if tp.dtype == np.uint16 else "f32"
    want = np.uint16 if dtype == "bf16" else np.float32
    if tp.dtype != want or tl.dtype != want:
        raise TypeError("parameter arrays do not match dtype")
    M, ld = tp.shape
    P = ld if P is None else P
    cd = np.zeros((num_cd(mix1, mix2), M), dtype=np.float64)
    c1, c2 = mix1.c(), mix2.c()
    seg = subset_array(subset)
    opts = _Opts(float(lr), float(mu), 1 if nesterov else 0, 1 if mix1_state else 0,
                 0 if seg is None else seg.shape[0], _ptr(seg))
    rc = lib().fgdo_outer_step(M, P, ld, 1 if dtype == "bf16" else 0, _ptr(tp), _ptr(tl), _ptr(v),
                               ctypes.byref(c1), ctypes.byref(c2), ctypes.byref(opts), _ptr(cd))
    if rc:
        raise ValueError(f"oracle outer step failed (rc={rc})")
    return tp, v, cd


def mix1_split(theta_prev, mix1: Mix, mom=None, mix1_state=False, P=None, dtype=None):
    """First half of split execution: returns (x stored in the parameter type,
    momentum after the optional state mix (a copy), cd[K1 + 1, M])."""
    tp = np.ascontiguousarray(theta_prev)
    if dtype is None:
        dtype = "bf16" if tp.dtype == np.uint16 else "f32"
    M, ld = tp.shape
    P = ld if P is None else P
    x = np.array(tp, copy=True)  # same type and shape; every [0, P) entry is overwritten
    v = None if mom is None else np.array(mom, dtype=np.float32, copy=True, order="C")
    cd = np.zeros((mix1.effective_rounds() + 1, M), dtype=np.float64)
    c1 = mix1.c()
    rc = lib().fgdo_mix1_split(M, P, ld, 1 if dtype == "bf16" else 0, _ptr(tp), _ptr(x), _ptr(v), ctypes.byref(c1),
                               1 if mix1_state else 0, _ptr(cd))
    if rc:
        raise ValueError(f"oracle Mix1 failed (rc={rc})")
    return x, v, cd


def outer_blocking(x, theta_prev, theta_local, mom, mix2: Mix, lr=0.7, mu=0.9, P=None, dtype=None, nesterov=True,
                   subset=None, write_local=False):
    """Second half of split execution.  Returns copies (theta', theta_local
    after the optional write-back, v', cd[K2 + 2, M])."""
    tp = np.array(theta_prev, copy=True, order="C")
    tl = np.array(theta_local, copy=True, order="C")
    xx = np.ascontiguousarray(x)
    v = np.array(mom, dtype=np.float32, copy=True, order="C")
    if dtype is None:
        dtype = "bf16" if tp.dtype == np.uint16 else "f32"
    M, ld = tp.shape
    P = ld if P is None else P
    cd = np.zeros((mix2.effective_rounds() + 2, M), dtype=np.float64)
    c2 = mix2.c()
    seg = subset_array(subset)
    opts = _Opts(float(lr), float(mu), 1 if nesterov else 0, 0, 0 if seg is None else seg.shape[0], _ptr(seg))
    rc = lib().fgdo_outer_blocking(M, P, ld, 1 if dtype == "bf16" else 0, _ptr(xx), _ptr(tp), _ptr(tl), _ptr(v),
                                   ctypes.byref(c2), ctypes.byref(opts), 1 if write_local else 0, _ptr(cd))
    if rc:
        raise ValueError(f"oracle blocking step failed (rc={rc})")
    return tp, tl, v, cd


def consensus(x, P=None, dtype=None):
    """S_m of a stored [M][ld] array.  Returns double[M]."""
    x = np.ascontiguousarray(x)
    if dtype is None:
        dtype = "bf16" if x.dtype == np.uint16 else "f32"
    M, ld = x.shape
    P = ld if P is None else P
    S = np.zeros(M, dtype=np.float64)
    rc = lib().fgdo_consensus(M, P, ld, 1 if dtype == "bf16" else 0, _ptr(x), _ptr(S))
    if rc:
        raise ValueError(f"oracle consensus failed (rc={rc})")
    return S
