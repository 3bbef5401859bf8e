"""Calls captured in a HIP graph (torch.cuda.graph) and replayed.

The JS distance enqueues kernels only (no allocation, copy or memset), and a
fused step whose topology is already on the device enqueues only its step
kernel and the consensus finalize, so both can sit in a graph, as a serving
loop or a caller that may not allocate would use them.  Each test replays
the graph several times, with eager work and synchronisations between the
replays, and checks every replay against the eager call bit for bit (the
kernels are deterministic).
"""

import numpy as np
import pytest

from synth import logits as slog
from synth import tensors
from tests import _parity as pa

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def env():
    import torch

    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    import paper_2606_22768_amd as fgd

    return fgd, torch


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_js_call_in_a_graph(env, dtype):
    fgd, torch = env
    M, U, K, k = 3, 40, 5003, 100
    ldk = -(-K // 8) * 8
    print(f"[graph] js {dtype} M={M} U={U} K={K}", flush=True)
    A, W = slog.numpy_logits(M, U, K, ldk, dtype, seed=5)
    conv = (lambda x: torch.from_numpy(x.view(np.int16)).cuda().view(torch.bfloat16)) if dtype == "bf16" \
        else (lambda x: torch.from_numpy(x).cuda())
    gA, gW = conv(A), conv(W)
    ws = torch.full((fgd.fgd_js_workspace_size(dtype, M, U),), 0xA5, dtype=torch.uint8, device="cuda")

    def outputs():
        return (torch.full((M, U), float("nan"), dtype=torch.float64, device="cuda"),
                torch.full((M,), float("nan"), dtype=torch.float64, device="cuda"),
                torch.full((U, k), -1, dtype=torch.int32, device="cuda"))

    d0, m0, t0 = outputs()
    fgd.fgd_js_distance(gA, gW, dtype, M, U, K, ldk, k, d0, m0, t0, ws)
    torch.cuda.synchronize()
    assert torch.isfinite(d0).all() and (t0 >= 0).all()

    d, m, t = outputs()
    s = torch.cuda.Stream()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        fgd.fgd_js_distance(gA, gW, dtype, M, U, K, ldk, k, d, m, t, ws)
    torch.cuda.synchronize()
    for rep in range(3):
        d.fill_(float("nan"))
        m.fill_(float("nan"))
        t.fill_(-1)
        ws.fill_(0x5A + rep)  # the workspace holds nothing from one call to the next
        fgd.fgd_js_distance(gA, gW, dtype, M, U, K, ldk, k, d0, m0, t0, ws)  # eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(d, d0) and torch.equal(m, m0) and torch.equal(t, t0), f"replay {rep}"


def test_fused_step_in_a_graph(env):
    fgd, torch = env
    M, P, dtype = 8, 5003, "bf16"
    ld = pa.aligned_ld(P)
    print(f"[graph] step M={M} P={P} {dtype}", flush=True)
    tp, tl, v = tensors.numpy_inputs(M, P, ld=ld, dtype=dtype, mom_std=1e-4, seed=3)
    t1 = pa.topo(("global",), M, 1)
    t2 = pa.topo(("ring", "metropolis", 0.1), M, 2, seed=11)
    dev = torch.device("cuda:0")

    def state():
        g_tp = torch.from_numpy(tp.view(np.int16)).to(dev).view(torch.bfloat16)
        g_tl = torch.from_numpy(tl.view(np.int16)).to(dev).view(torch.bfloat16)
        return g_tp, g_tl, torch.from_numpy(v).to(dev)

    eng = fgd.Engine(M, P, ld, dtype, 0.7, 0.9, device=0)
    try:
        eng.set_topology_dict("mix1", t1)
        eng.set_topology_dict("mix2", t2)
        s = torch.cuda.Stream()
        ea, eb = state(), state()  # eager copy, graph copy
        cd_a = torch.full((eng.num_cd_rows(), M), float("nan"), dtype=torch.float64, device=dev)
        cd_b = torch.full_like(cd_a, float("nan"))
        # The first eager step uploads the topology on stream s; the capture
        # on s then holds the step kernel and the finalize only.
        eng.outer_step(*ea, cd_a, stream=s)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s):
            eng.outer_step(*eb, cd_b, stream=s)
        torch.cuda.synchronize()
        for rep in range(3):
            if rep > 0:
                eng.outer_step(*ea, cd_a, stream=s)  # eager step rep + 1 on the eager copy
            cd_b.fill_(float("nan"))
            torch.cuda.synchronize()
            g.replay()  # step rep + 1 on the graph copy
            torch.cuda.synchronize()
            assert torch.equal(eb[0].view(torch.int16), ea[0].view(torch.int16)), f"theta after replay {rep}"
            assert torch.equal(eb[2], ea[2]), f"momentum after replay {rep}"
            assert torch.equal(cd_b, cd_a), f"consensus after replay {rep}"
        assert torch.equal(eb[1].view(torch.int16), ea[1].view(torch.int16))  # theta_local is only read
    finally:
        eng.close()
