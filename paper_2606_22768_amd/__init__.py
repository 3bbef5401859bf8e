"""Python binding of libfgd (include/fgd.h): the fused Factored Gossip DiLoCo
outer step for AMD MI355X.

Every function here has the name of the C entry point it wraps and only
marshals arguments: numpy arrays become host pointers, torch tensors become
device pointers, and the current torch stream becomes the hipStream_t.  All
arithmetic of the step runs in the library's HIP kernels.  If libfgd.so has
not been built, importing this package raises ImportError.
"""

from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libfgd.so")

FGD_OK, FGD_ERR_INVALID_ARG, FGD_ERR_TOPOLOGY, FGD_ERR_UNSUPPORTED = 0, 1, 2, 3
FGD_ERR_OUT_OF_MEMORY, FGD_ERR_HIP, FGD_ERR_STATE = 4, 5, 6
FGD_F32, FGD_BF16 = 0, 1
FGD_MIX1, FGD_MIX2 = 1, 2
FGD_W_IDENTITY, FGD_W_GLOBAL_MEAN, FGD_W_CSR = 0, 1, 2
FGD_REWEIGHT_NONE, FGD_REWEIGHT_METROPOLIS, FGD_REWEIGHT_SELF = 0, 1, 2
FGD_MAX_WORKERS, FGD_MAX_ROUNDS, FGD_MAX_SUBSET_SEGMENTS = 64, 8, 4096
FGD_MAX_JS_TOPK, FGD_MAX_JS_WORKERS = 1024, 4096

DTYPES = {"f32": FGD_F32, "bf16": FGD_BF16}
KINDS = {"identity": FGD_W_IDENTITY, "global": FGD_W_GLOBAL_MEAN, "csr": FGD_W_CSR}
REWEIGHTS = {"none": FGD_REWEIGHT_NONE, "metropolis": FGD_REWEIGHT_METROPOLIS, "self": FGD_REWEIGHT_SELF}
MIXES = {"mix1": FGD_MIX1, "mix2": FGD_MIX2, 1: FGD_MIX1, 2: FGD_MIX2}


class FgdError(RuntimeError):
    def __init__(self, status: int, where: str, detail: str):
        super().__init__(f"{where}: {fgd_status_string(status)}: {detail}")
        self.status = status


class fgd_config(ctypes.Structure):
    _fields_ = [("struct_size", ctypes.c_uint32), ("num_workers", ctypes.c_int32),
                ("num_params", ctypes.c_int64), ("ld", ctypes.c_int64), ("param_dtype", ctypes.c_int32),
                ("state_dtype", ctypes.c_int32), ("outer_lr", ctypes.c_float), ("momentum", ctypes.c_float),
                ("nesterov", ctypes.c_int32), ("device", ctypes.c_int32), ("mix1_state", ctypes.c_int32),
                ("reserved", ctypes.c_int32)]


def _load():
    # PyTorch supplies device memory and streams.  Its HIP runtime and the one
    # libfgd.so links against share the soname libamdhip64.so.7; loading torch
    # first makes the dynamic loader bind libfgd.so to torch's copy, so one
    # runtime serves both and torch stream handles are valid here.
    import torch  # noqa: F401

    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with `python paper_2606_22768_amd/build.py`")
    L = ctypes.CDLL(LIB_PATH)
    P, I32, I64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    sig = {
        "fgd_create": (I32, [ctypes.POINTER(fgd_config), ctypes.POINTER(ctypes.c_void_p)]),
        "fgd_destroy": (I32, [P]),
        "fgd_set_topology": (I32, [P, I32, I32, P, P, P, I32, P, I32]),
        "fgd_set_mix2_subset": (I32, [P, P, I32]),
        "fgd_num_cd_rows": (I32, [P, ctypes.POINTER(I32)]),
        "fgd_step_variant": (I32, [P, ctypes.POINTER(I32)]),
        "fgd_outer_step": (I32, [P, P, P, P, P, P]),
        "fgd_mix1": (I32, [P, P, P, P, P, I32, P]),
        "fgd_outer_step_blocking": (I32, [P, P, P, P, P, P, I32, P]),
        "fgd_num_cd_rows_split": (I32, [P, ctypes.POINTER(I32), ctypes.POINTER(I32)]),
        "fgd_min_bytes_split": (I32, [P, I32, ctypes.POINTER(I64), ctypes.POINTER(I64)]),
        "fgd_consensus_distance": (I32, [P, P, I32, P, P]),
        "fgd_consensus_distance_noalloc": (I32, [I32, I64, I64, I32, P, P, P]),
        "fgd_get_effective_weights": (I32, [P, I32, I32, P]),
        "fgd_effective_weights": (I32, [I32, P, P, P, P, I32, P]),
        "fgd_min_bytes_per_step": (I32, [P, ctypes.POINTER(I64)]),
        "fgd_state_layout": (I32, [P, I32, I32, I64, ctypes.POINTER(I64), ctypes.POINTER(I64)]),
        "fgd_enable_timing": (I32, [P, I32]),
        "fgd_read_timing": (I32, [P, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(I64)]),
        "fgd_stream_copy": (I32, [P, P, I64, P]),
        "fgd_stream_step_pattern": (I32, [P, P, P, P, P]),
        "fgd_js_distance": (I32, [P, P, I32, I32, I64, I64, I64, I32, P, P, P, P, I64, P]),
        "fgd_js_workspace_size": (I32, [I32, I32, I64, ctypes.POINTER(I64)]),
        "fgd_stream_js_pattern": (I32, [P, P, I32, I32, I64, I64, I64, P, I64, P]),
        "fgd_status_string": (ctypes.c_char_p, [I32]),
        "fgd_last_error": (ctypes.c_char_p, []),
        "fgd_source_hash": (ctypes.c_char_p, [I32]),
    }
    for name, (res, args) in sig.items():
        f = getattr(L, name)
        f.restype, f.argtypes = res, args
    _check_sources(L)
    return L


def _library_hashes(L):
    return {c: L.fgd_source_hash(i).decode() for i, c in enumerate(("all", "step", "js"))}


def _check_sources(L, root=None):
    """Refuses a library built from other sources than the tree beside it:
    its tests and timings would describe other code."""
    from . import build as _build

    root = root or _build.ROOT
    if not os.path.isdir(os.path.join(root, "paper_2606_22768_amd", "csrc")):
        return  # an installed copy without sources: nothing to compare with
    have, want = _library_hashes(L), _build.source_hashes(root)
    if have["all"] != want["all"]:
        raise ImportError(f"{LIB_PATH} was built from other sources (library {have['all']}, sources "
                          f"{want['all']}): rebuild it with `python paper_2606_22768_amd/build.py`")


lib = _load()


def library_source_hash() -> dict:
    """The source hashes compiled into the loaded library (all, step, js)."""
    return _library_hashes(lib)


def fgd_status_string(status: int) -> str:
    return lib.fgd_status_string(int(status)).decode()


def fgd_last_error() -> str:
    return lib.fgd_last_error().decode()


def _check(status: int, where: str):
    if status != FGD_OK:
        raise FgdError(status, where, fgd_last_error())


def _host(a, dtype):
    """Contiguous numpy copy (kept alive by the caller) and its address, or (None, None)."""
    if a is None:
        return None, None
    arr = np.ascontiguousarray(a, dtype=dtype)
    return arr, arr.ctypes.data


def _dev(t):
    """Device address of a torch tensor (or an int address), None for None."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    if not t.is_cuda:
        raise ValueError("expected a device tensor")
    return t.data_ptr()


def _stream(stream):
    if stream is None:
        import torch

        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


# --------------------------------------------------------------- raw C ABI

def fgd_create(num_workers, num_params, ld=None, param_dtype="f32", outer_lr=0.7, momentum=0.9, device=0,
               nesterov=True, mix1_state=False, state_dtype="f32"):
    cfg = fgd_config(ctypes.sizeof(fgd_config), int(num_workers), int(num_params),
                     int(num_params if ld is None else ld), DTYPES.get(param_dtype, param_dtype),
                     DTYPES.get(state_dtype, state_dtype), float(outer_lr), float(momentum),
                     int(nesterov), int(device), int(mix1_state), 0)
    h = ctypes.c_void_p()
    _check(lib.fgd_create(ctypes.byref(cfg), ctypes.byref(h)), "fgd_create")
    return h


def fgd_destroy(h):
    _check(lib.fgd_destroy(h), "fgd_destroy")


def fgd_set_topology(h, which, kind, row_ptr=None, col_idx=None, weights=None, num_rounds=0, edge_masks=None,
                     reweight="none"):
    rp, prp = _host(row_ptr, np.int32)
    ci, pci = _host(col_idx, np.int32)
    w, pw = _host(weights, np.float32)
    mk, pmk = _host(edge_masks, np.uint8)
    _check(lib.fgd_set_topology(h, MIXES[which], KINDS.get(kind, kind), prp, pci, pw, int(num_rounds), pmk,
                                REWEIGHTS.get(reweight, reweight)), "fgd_set_topology")


def fgd_set_mix2_subset(h, segments=None):
    """segments: [n][2] int64 half-open parameter ranges, or None / empty for no subset."""
    seg = None if segments is None else np.ascontiguousarray(np.asarray(segments, dtype=np.int64).reshape(-1, 2))
    n = 0 if seg is None else seg.shape[0]
    _check(lib.fgd_set_mix2_subset(h, seg.ctypes.data if n else None, n), "fgd_set_mix2_subset")


def fgd_num_cd_rows(h) -> int:
    n = ctypes.c_int32()
    _check(lib.fgd_num_cd_rows(h, ctypes.byref(n)), "fgd_num_cd_rows")
    return n.value


FGD_STEP_LANE_PER_PARAM, FGD_STEP_WORKER_GROUPS = 0, 1


def fgd_step_variant(h) -> int:
    n = ctypes.c_int32()
    _check(lib.fgd_step_variant(h, ctypes.byref(n)), "fgd_step_variant")
    return n.value


def fgd_outer_step(h, theta_prev, theta_local, momentum, cd_out=None, stream=None):
    _check(lib.fgd_outer_step(h, _dev(theta_prev), _dev(theta_local), _dev(momentum), _dev(cd_out),
                              _stream(stream)), "fgd_outer_step")


def fgd_mix1(h, theta_prev, x_out, momentum=None, cd_out=None, num_blocks=0, stream=None):
    _check(lib.fgd_mix1(h, _dev(theta_prev), _dev(x_out), _dev(momentum), _dev(cd_out), int(num_blocks),
                        _stream(stream)), "fgd_mix1")


def fgd_outer_step_blocking(h, x, theta_prev, theta_local, momentum, cd_out=None, write_local=False, stream=None):
    _check(lib.fgd_outer_step_blocking(h, _dev(x), _dev(theta_prev), _dev(theta_local), _dev(momentum),
                                       _dev(cd_out), 1 if write_local else 0, _stream(stream)),
           "fgd_outer_step_blocking")


def fgd_num_cd_rows_split(h):
    a, b = ctypes.c_int32(), ctypes.c_int32()
    _check(lib.fgd_num_cd_rows_split(h, ctypes.byref(a), ctypes.byref(b)), "fgd_num_cd_rows_split")
    return a.value, b.value


def fgd_min_bytes_split(h, write_local=False):
    a, b = ctypes.c_int64(), ctypes.c_int64()
    _check(lib.fgd_min_bytes_split(h, 1 if write_local else 0, ctypes.byref(a), ctypes.byref(b)),
           "fgd_min_bytes_split")
    return a.value, b.value


def fgd_consensus_distance(h, x, dtype, out, stream=None):
    _check(lib.fgd_consensus_distance(h, _dev(x), DTYPES.get(dtype, dtype), _dev(out), _stream(stream)),
           "fgd_consensus_distance")


def fgd_consensus_distance_noalloc(num_workers, num_params, ld, dtype, x, out, stream=None):
    _check(lib.fgd_consensus_distance_noalloc(int(num_workers), int(num_params), int(ld), DTYPES.get(dtype, dtype),
                                              _dev(x), _dev(out), _stream(stream)), "fgd_consensus_distance_noalloc")


def fgd_get_effective_weights(h, which, rnd, nnz):
    out = np.zeros(int(nnz), dtype=np.float32)
    _check(lib.fgd_get_effective_weights(h, MIXES[which], int(rnd), out.ctypes.data), "fgd_get_effective_weights")
    return out


def fgd_effective_weights(num_workers, row_ptr, col_idx, weights=None, mask=None, reweight="none"):
    rp, prp = _host(row_ptr, np.int32)
    ci, pci = _host(col_idx, np.int32)
    w, pw = _host(weights, np.float32)
    mk, pmk = _host(mask, np.uint8)
    out = np.zeros(0 if ci is None else ci.shape[0], dtype=np.float32)
    _check(lib.fgd_effective_weights(int(num_workers), prp, pci, pw, pmk, REWEIGHTS.get(reweight, reweight),
                                     out.ctypes.data if out.size else None), "fgd_effective_weights")
    return out


def fgd_min_bytes_per_step(h) -> int:
    b = ctypes.c_int64()
    _check(lib.fgd_min_bytes_per_step(h, ctypes.byref(b)), "fgd_min_bytes_per_step")
    return b.value


def fgd_state_layout(h, spread=True, with_x=False, range_bytes=0):
    """Returns ((theta_prev, theta_local, x, momentum) byte offsets, total bytes);
    the x offset is -1 without x."""
    offs, total = (ctypes.c_int64 * 4)(), ctypes.c_int64()
    _check(lib.fgd_state_layout(h, 1 if spread else 0, 1 if with_x else 0, int(range_bytes), offs,
                                ctypes.byref(total)), "fgd_state_layout")
    return tuple(offs), total.value


def fgd_enable_timing(h, enable=True):
    _check(lib.fgd_enable_timing(h, 1 if enable else 0), "fgd_enable_timing")


def fgd_read_timing(h):
    ms, n = ctypes.c_double(), ctypes.c_int64()
    _check(lib.fgd_read_timing(h, ctypes.byref(ms), ctypes.byref(n)), "fgd_read_timing")
    return ms.value, n.value


def fgd_js_workspace_size(dtype, num_workers, num_tokens) -> int:
    n = ctypes.c_int64()
    _check(lib.fgd_js_workspace_size(DTYPES.get(dtype, dtype), int(num_workers), int(num_tokens), ctypes.byref(n)),
           "fgd_js_workspace_size")
    return n.value


def fgd_js_distance(logits_avg, logits_workers, dtype, num_workers, num_tokens, vocab, ldk, top_k, d_out,
                    mean_out=None, topk_out=None, workspace=None, workspace_bytes=None, stream=None):
    """The C call; `workspace` is device memory of at least
    fgd_js_workspace_size bytes (a tensor's size is taken when
    workspace_bytes is None)."""
    if workspace_bytes is None:
        workspace_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib.fgd_js_distance(_dev(logits_avg), _dev(logits_workers), DTYPES.get(dtype, dtype), int(num_workers),
                               int(num_tokens), int(vocab), int(ldk), int(top_k), _dev(d_out), _dev(mean_out),
                               _dev(topk_out), _dev(workspace), int(workspace_bytes), _stream(stream)),
           "fgd_js_distance")


def fgd_stream_js_pattern(logits_avg, logits_workers, dtype, num_workers, num_tokens, vocab, ldk, workspace,
                          workspace_bytes=None, stream=None):
    """The JS row kernel's loads without its arithmetic (a streaming
    reference); same arguments as fgd_js_distance's logits and workspace."""
    if workspace_bytes is None:
        workspace_bytes = workspace.numel() * workspace.element_size()
    _check(lib.fgd_stream_js_pattern(_dev(logits_avg), _dev(logits_workers), DTYPES.get(dtype, dtype),
                                     int(num_workers), int(num_tokens), int(vocab), int(ldk), _dev(workspace),
                                     int(workspace_bytes), _stream(stream)), "fgd_stream_js_pattern")


def js_distance(logits_avg, logits_workers, top_k=100, vocab=None, d_out=None, mean_out=None, topk_out=None,
                workspace=None, stream=None):
    """Tensor-level call: logits_avg [U][ldk], logits_workers [M][U][ldk]
    (float32 or bfloat16, rows contiguous); returns (d [M][U], mean [M]).
    The workspace (a uint8 device tensor) is allocated when not given."""
    import torch

    dtype = {torch.float32: "f32", torch.bfloat16: "bf16"}[logits_avg.dtype]
    if logits_workers.dtype != logits_avg.dtype:
        raise TypeError("logits_avg and logits_workers must share a dtype")
    U, ldk = logits_avg.shape
    M = logits_workers.shape[0]
    if tuple(logits_workers.shape) != (M, U, ldk) or not logits_workers.is_contiguous() \
            or not logits_avg.is_contiguous():
        raise ValueError("expected contiguous logits_avg [U][ldk] and logits_workers [M][U][ldk]")
    K = ldk if vocab is None else int(vocab)
    # The kernels write through the raw pointers, so a caller's buffer of
    # another dtype, a smaller one or a non-contiguous one is refused here,
    # before anything is enqueued; then every tensor must share the logits'
    # GPU.
    _check_js_buffer(d_out, "d_out", torch.float64, M * U)
    _check_js_buffer(mean_out, "mean_out", torch.float64, M)
    _check_js_buffer(topk_out, "topk_out", torch.int32, U * int(top_k))
    need_ws = fgd_js_workspace_size(dtype, M, U)
    _check_js_buffer(workspace, "workspace", None, need_ws)
    dev = logits_avg.device
    for name, t in (("logits_avg", logits_avg), ("logits_workers", logits_workers), ("d_out", d_out),
                    ("mean_out", mean_out), ("topk_out", topk_out), ("workspace", workspace)):
        if t is not None and (not t.is_cuda or t.device != dev):
            raise ValueError(f"{name}: expected a tensor on the logits' GPU, got {t.device}")
    d_out = torch.empty((M, U), dtype=torch.float64, device=dev) if d_out is None else d_out
    mean_out = torch.empty(M, dtype=torch.float64, device=dev) if mean_out is None else mean_out
    if workspace is None:
        workspace = torch.empty(need_ws, dtype=torch.uint8, device=dev)
    fgd_js_distance(logits_avg, logits_workers, dtype, M, U, K, ldk, top_k, d_out, mean_out, topk_out, workspace,
                    None, stream)
    return d_out, mean_out


def _check_js_buffer(t, name, dtype, need):
    """A caller-supplied js_distance buffer: a contiguous tensor of `dtype`
    (any dtype when None) holding at least `need` elements (bytes when dtype
    is None)."""
    import torch

    if t is None:
        return
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name}: expected a torch tensor, got {type(t).__name__}")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name}: expected {dtype}, got {t.dtype}")
    size = t.numel() if dtype is not None else t.numel() * t.element_size()
    if size < need:
        unit = "elements" if dtype is not None else "bytes"
        raise ValueError(f"{name}: needs at least {need} {unit}, got {size}")
    if not t.is_contiguous():
        raise ValueError(f"{name}: must be contiguous")


def fgd_stream_step_pattern(h, theta_prev, theta_local, momentum, stream=None):
    _check(lib.fgd_stream_step_pattern(h, _dev(theta_prev), _dev(theta_local), _dev(momentum), _stream(stream)),
           "fgd_stream_step_pattern")


def fgd_stream_copy(dst, src, nbytes, stream=None):
    _check(lib.fgd_stream_copy(_dev(dst), _dev(src), int(nbytes), _stream(stream)), "fgd_stream_copy")


# ------------------------------------------------------ tensor-level wrapper

class Engine:
    """One engine over M worker rows of P parameters stored [M][ld].

    Methods map one-to-one onto the C entry points; they only check that
    tensors have the layout the engine was created for.
    """

    def __init__(self, num_workers, num_params, ld=None, param_dtype="f32", outer_lr=0.7, momentum=0.9, device=0,
                 nesterov=True, mix1_state=False):
        self.M, self.P = int(num_workers), int(num_params)
        self.ld = self.P if ld is None else int(ld)
        self.dtype = param_dtype
        self.device = device
        self.handle = fgd_create(self.M, self.P, self.ld, param_dtype, outer_lr, momentum, device, nesterov,
                                 mix1_state)
        self._nnz = {1: 0, 2: 0}

    def close(self):
        if self.handle is not None:
            fgd_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def set_topology(self, which, kind, row_ptr=None, col_idx=None, weights=None, rounds=0, masks=None,
                     reweight="none"):
        fgd_set_topology(self.handle, which, kind, row_ptr, col_idx, weights, rounds, masks, reweight)
        self._nnz[MIXES[which]] = 0 if col_idx is None else len(col_idx)

    def set_topology_dict(self, which, t):
        """From the dict produced by synth.configs.topology."""
        self.set_topology(which, t["kind"], t["row_ptr"], t["col_idx"], t["weights"], t["rounds"], t["masks"],
                          t["reweight"])

    def set_mix2_subset(self, segments=None):
        fgd_set_mix2_subset(self.handle, segments)

    def num_cd_rows(self):
        return fgd_num_cd_rows(self.handle)

    def step_variant(self):
        """"worker-groups" or "lane-per-param": the kernel fgd_outer_step launches."""
        return "worker-groups" if fgd_step_variant(self.handle) == FGD_STEP_WORKER_GROUPS else "lane-per-param"

    def _check_rows(self, t, name, dtype):
        import torch

        want = {"f32": torch.float32, "bf16": torch.bfloat16}[dtype]
        if t.dtype != want:
            raise TypeError(f"{name}: expected {want}, got {t.dtype}")
        if t.dim() != 2 or t.shape[0] != self.M or t.shape[1] < self.P:
            raise ValueError(f"{name}: expected shape [{self.M}, >= {self.P}], got {tuple(t.shape)}")
        if t.stride(1) != 1 or (self.M > 1 and t.stride(0) != self.ld):
            raise ValueError(f"{name}: rows must be contiguous with row stride ld = {self.ld}")
        if not t.is_cuda or t.device.index != self.device:
            raise ValueError(f"{name}: expected a tensor on cuda:{self.device}, got {t.device}")

    def _check_out(self, t, name, rows):
        """A consensus output: float64, rows x M doubles or more, contiguous, on
        the engine's device.  The kernels write rows * M doubles through the
        raw pointer, so a smaller or differently typed buffer is refused here,
        before anything is enqueued."""
        import torch

        if t is None:
            return
        if not isinstance(t, torch.Tensor):
            raise TypeError(f"{name}: expected a torch tensor, got {type(t).__name__}")
        if t.dtype != torch.float64:
            raise TypeError(f"{name}: expected torch.float64, got {t.dtype}")
        need = int(rows) * self.M
        if t.numel() < need:
            raise ValueError(f"{name}: needs at least {rows} x {self.M} = {need} doubles, got {t.numel()}")
        if not t.is_contiguous():
            raise ValueError(f"{name}: must be contiguous")
        if not t.is_cuda or t.device.index != self.device:
            raise ValueError(f"{name}: expected a tensor on cuda:{self.device}, got {t.device}")

    def _stream(self, stream):
        """The given stream, or torch's current stream on the engine's device."""
        if stream is not None:
            return stream
        import torch

        return torch.cuda.current_stream(self.device)

    def outer_step(self, theta_prev, theta_local, momentum, cd_out=None, stream=None):
        if cd_out is not None:
            self._check_out(cd_out, "cd_out", self.num_cd_rows())
        self._check_rows(theta_prev, "theta_prev", self.dtype)
        self._check_rows(theta_local, "theta_local", self.dtype)
        self._check_rows(momentum, "momentum", "f32")
        fgd_outer_step(self.handle, theta_prev, theta_local, momentum, cd_out, self._stream(stream))

    def mix1(self, theta_prev, x_out, momentum=None, cd_out=None, stream=None, num_blocks=0):
        """Mix1 half of split execution: x_out = Mix1(theta_prev) (and the
        momentum mixed in place when the engine mixes the state)."""
        if cd_out is not None:
            self._check_out(cd_out, "cd_out", self.num_cd_rows_split()[0])
        self._check_rows(theta_prev, "theta_prev", self.dtype)
        self._check_rows(x_out, "x_out", self.dtype)
        if momentum is not None:
            self._check_rows(momentum, "momentum", "f32")
        fgd_mix1(self.handle, theta_prev, x_out, momentum, cd_out, num_blocks, self._stream(stream))

    def outer_step_blocking(self, x, theta_prev, theta_local, momentum, cd_out=None, write_local=False, stream=None):
        """Blocking half of split execution, from the stored Mix1 output x."""
        if cd_out is not None:
            self._check_out(cd_out, "cd_out", self.num_cd_rows_split()[1])
        self._check_rows(x, "x", self.dtype)
        self._check_rows(theta_prev, "theta_prev", self.dtype)
        self._check_rows(theta_local, "theta_local", self.dtype)
        self._check_rows(momentum, "momentum", "f32")
        fgd_outer_step_blocking(self.handle, x, theta_prev, theta_local, momentum, cd_out, write_local,
                                self._stream(stream))

    def num_cd_rows_split(self):
        return fgd_num_cd_rows_split(self.handle)

    def min_bytes_split(self, write_local=False):
        return fgd_min_bytes_split(self.handle, write_local)

    def consensus_distance(self, x, out, stream=None, dtype=None):
        dtype = dtype or self.dtype
        self._check_out(out, "out", 1)
        self._check_rows(x, "x", dtype)
        fgd_consensus_distance(self.handle, x, dtype, out, self._stream(stream))

    def effective_weights(self, which, rnd):
        return fgd_get_effective_weights(self.handle, which, rnd, self._nnz[MIXES[which]])

    def min_bytes_per_step(self):
        return fgd_min_bytes_per_step(self.handle)

    def state_layout(self, spread=True, with_x=False, range_bytes=0):
        return fgd_state_layout(self.handle, spread, with_x, range_bytes)

    def alloc_state(self, spread=True, with_x=False, range_bytes=0):
        """One device buffer laid out by fgd_state_layout and [M][ld] views of
        it: dict(pool, theta_prev, theta_local, x (or None), momentum, offsets),
        offsets being the layout's byte offsets.  The views share the pool's
        memory; their contents are uninitialised."""
        import torch

        offs, total = self.state_layout(spread, with_x, range_bytes)
        pool = torch.empty(total, dtype=torch.uint8, device=f"cuda:{self.device}")
        pdt = {"f32": torch.float32, "bf16": torch.bfloat16}[self.dtype]
        es = 4 if self.dtype == "f32" else 2

        def view(off, dt, size):
            return pool[off:off + self.M * self.ld * size].view(dt).view(self.M, self.ld)

        return {"pool": pool, "theta_prev": view(offs[0], pdt, es), "theta_local": view(offs[1], pdt, es),
                "x": None if offs[2] < 0 else view(offs[2], pdt, es),
                "momentum": view(offs[3], torch.float32, 4), "offsets": offs}

    def stream_step_pattern(self, theta_prev, theta_local, momentum, stream=None):
        """The step's memory traffic without its arithmetic (arrays unchanged)."""
        self._check_rows(theta_prev, "theta_prev", self.dtype)
        self._check_rows(theta_local, "theta_local", self.dtype)
        self._check_rows(momentum, "momentum", "f32")
        fgd_stream_step_pattern(self.handle, theta_prev, theta_local, momentum, self._stream(stream))

    def enable_timing(self, on=True):
        fgd_enable_timing(self.handle, on)

    def read_timing(self):
        return fgd_read_timing(self.handle)
