"""GPU: the step on arrays placed by fgd_state_layout (one buffer, the
momentum one physical-memory range past the parameter arrays, or packed)
matches the oracle, and the split halves run on the x the layout places.
Every call goes through the C ABI (libfgd.so).
"""

import numpy as np
import pytest

import oracle
from synth import configs, tensors
from tests import _parity as pa

pytestmark = pytest.mark.gpu

GiB = 1 << 30


@pytest.fixture(scope="module")
def env():
    import torch

    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    import paper_2606_22768_amd as fgd

    return fgd, torch


def _to_dev(torch, a, dtype, out):
    src = torch.from_numpy(a) if dtype == "f32" or a.dtype == np.float32 else \
        torch.from_numpy(a.view(np.int16)).view(torch.bfloat16)
    out.copy_(src.to(out.device))


def _from_dev(t, dtype):
    c = t.cpu()
    return c.numpy() if dtype == "f32" else c.view(__import__("torch").int16).numpy().view(np.uint16)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("spread", [True, False])
def test_step_on_state_layout(env, dtype, spread):
    fgd, torch = env
    M, P = 8, 3 * 1024 + 5
    ld = pa.aligned_ld(P)
    print(f"[layout] dtype={dtype} spread={spread} M={M} P={P}", flush=True)
    tp, tl, v = tensors.numpy_inputs(M, P, ld=ld, dtype=dtype, seed=5)
    t1 = configs.topology(("global",), M, 1, 0)
    t2 = configs.topology(("ring", "metropolis", 0.1), M, 1, 0, step=3)
    ref_t, ref_v, ref_cd = oracle.outer_step(tp, tl, v, oracle.Mix.from_topology(t1), oracle.Mix.from_topology(t2),
                                             P=P, dtype=dtype)
    eng = fgd.Engine(M, P, ld, dtype, device=0)
    try:
        eng.set_topology_dict("mix1", t1)
        eng.set_topology_dict("mix2", t2)
        st = eng.alloc_state(spread=spread, with_x=True)
        offs = st["offsets"]
        if spread:  # the range derived from the device: a third of its memory, whole GiB
            total_mem = torch.cuda.get_device_properties(0).total_memory
            assert offs[3] == (total_mem // 3 + GiB // 2) // GiB * GiB
        else:
            assert offs[3] == offs[2] + -(-M * ld * (2 if dtype == "bf16" else 4) // (2 << 20)) * (2 << 20)
        _to_dev(torch, tp, dtype, st["theta_prev"])
        _to_dev(torch, tl, dtype, st["theta_local"])
        st["momentum"].copy_(torch.from_numpy(v).to(st["momentum"].device))
        cd = torch.full((eng.num_cd_rows(), M), float("nan"), dtype=torch.float64, device="cuda:0")
        eng.outer_step(st["theta_prev"], st["theta_local"], st["momentum"], cd)
        torch.cuda.synchronize()
        got_t, got_v = _from_dev(st["theta_prev"], dtype), st["momentum"].cpu().numpy()
        scale = float(np.abs(tensors.bf16_bits_to_f32(tp) if dtype == "bf16" else tp).max())
        pa.compare_outputs(dtype, got_t, ref_t, got_v, ref_v, P, scale)
        pa.compare_step_cd(cd.cpu().numpy(), ref_cd, ref_t, dtype, P, scale)
        # The split halves on the same buffer: Mix1 into the placed x; then
        # the blocking half from the oracle's x, restarting from the inputs.
        _to_dev(torch, tp, dtype, st["theta_prev"])
        st["momentum"].copy_(torch.from_numpy(v).to(st["momentum"].device))
        eng.mix1(st["theta_prev"], st["x"])
        torch.cuda.synchronize()
        ref_x = oracle.mix1_split(tp, oracle.Mix.from_topology(t1), P=P, dtype=dtype)[0]
        got_x = _from_dev(st["x"], dtype)
        if dtype == "f32":
            assert pa.max_row_rel_err(got_x[:, :P], ref_x[:, :P]) <= 1e-6
        else:
            assert np.abs(pa.ordered_bf16(got_x[:, :P]) - pa.ordered_bf16(ref_x[:, :P])).max() <= 1
        _to_dev(torch, ref_x, dtype, st["x"])
        eng.outer_step_blocking(st["x"], st["theta_prev"], st["theta_local"], st["momentum"])
        torch.cuda.synchronize()
        ref_bt, _, ref_bv, _ = oracle.outer_blocking(ref_x, tp, tl, v, oracle.Mix.from_topology(t2), P=P, dtype=dtype)
        pa.compare_outputs(dtype, _from_dev(st["theta_prev"], dtype), ref_bt, st["momentum"].cpu().numpy(), ref_bv,
                           P, scale)
    finally:
        eng.close()
        del st
        torch.cuda.empty_cache()
