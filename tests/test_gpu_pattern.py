"""GPU: the access-pattern reference (fgd_stream_step_pattern) moves the
step's bytes but leaves every array bit-identical, on ragged sizes, both
storage types and every worker count it serves; it refuses the others.
Every call goes through the C ABI (libfgd.so)."""

import numpy as np
import pytest

from synth import tensors
from tests import _parity as pa

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def env():
    import torch

    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    import paper_2606_22768_amd as fgd

    return fgd, torch


@pytest.mark.parametrize("M,P,dtype", [(8, 3 * 1024 + 5, "bf16"), (8, 4096, "f32"), (16, 2049, "f32"),
                                       (64, 777, "f32"), (64, 300, "bf16"), (1, 17, "bf16"), (32, 1000, "f32")])
def test_pattern_leaves_arrays_unchanged(env, M, P, dtype):
    fgd, torch = env
    print(f"[pattern] M={M} P={P} {dtype}", flush=True)
    ld = pa.aligned_ld(P) + 8
    tp, tl, v = tensors.numpy_inputs(M, P, ld=ld, dtype=dtype, seed=M + P)
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    dev = lambda a, t: (torch.from_numpy(a).cuda() if a.dtype == np.float32 and t == torch.float32
                        else torch.from_numpy(a.view(np.int16)).cuda().view(t))
    g_tp, g_tl, g_v = dev(tp, tdt), dev(tl, tdt), torch.from_numpy(v).cuda()
    g_tp[0, 0] = float("-0.0")  # signed zero and non-finite values keep their bits too
    g_v[M - 1, P - 1] = float("nan")
    before = [t.clone() for t in (g_tp, g_tl, g_v)]
    eng = fgd.Engine(M, P, ld, dtype, device=0)
    try:
        for _ in range(2):
            eng.stream_step_pattern(g_tp, g_tl, g_v)
        torch.cuda.synchronize()
    finally:
        eng.close()
    for a, b in zip((g_tp, g_tl, g_v), before):
        w = torch.int16 if a.dtype == torch.bfloat16 else torch.int32
        assert torch.equal(a.view(w), b.view(w))


def test_pattern_refuses_other_worker_counts(env):
    fgd, torch = env
    eng = fgd.Engine(3, 64, 64, "f32", device=0)
    try:
        x = torch.zeros((3, 64), device="cuda")
        with pytest.raises(fgd.FgdError) as e:
            eng.stream_step_pattern(x, x.clone(), x.clone())
        assert e.value.status == fgd.FGD_ERR_UNSUPPORTED
    finally:
        eng.close()


@pytest.mark.parametrize("P,dtype", [(777, "f32"), (300, "bf16"), (300_001, "f32")])
def test_worker_group_pattern_leaves_arrays_unchanged(env, P, dtype):
    """With a topology that selects the 64-worker worker-group step, the
    reference follows that layout; it too leaves every array bit-identical."""
    fgd, torch = env
    M = 64
    print(f"[pattern wg] P={P} {dtype}", flush=True)
    ld = pa.aligned_ld(P) + 8
    tp, tl, v = tensors.numpy_inputs(M, P, ld=ld, dtype=dtype, seed=P)
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    dev = lambda a, t: (torch.from_numpy(a).cuda() if a.dtype == np.float32 and t == torch.float32
                        else torch.from_numpy(a.view(np.int16)).cuda().view(t))
    g_tp, g_tl, g_v = dev(tp, tdt), dev(tl, tdt), torch.from_numpy(v).cuda()
    g_v[M - 1, P - 1] = float("nan")
    before = [t.clone() for t in (g_tp, g_tl, g_v)]
    eng = fgd.Engine(M, P, ld, dtype, device=0)
    try:
        reg4 = ("regular", "metropolis", 4)
        eng.set_topology_dict("mix1", pa.topo(reg4, M, 1))
        eng.set_topology_dict("mix2", pa.topo(reg4, M, 3))
        assert eng.step_variant() == "worker-groups"
        for _ in range(2):
            eng.stream_step_pattern(g_tp, g_tl, g_v)
        torch.cuda.synchronize()
    finally:
        eng.close()
    for a, b in zip((g_tp, g_tl, g_v), before):
        w = torch.int16 if a.dtype == torch.bfloat16 else torch.int32
        assert torch.equal(a.view(w), b.view(w))
