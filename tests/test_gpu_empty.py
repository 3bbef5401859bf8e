"""Empty parameter vectors (P = 0) on every entry point that launches a
kernel: nothing is read or written, every consensus entry is 0, and the
call succeeds.  The fused step's own P = 0 case sits with the parity tests;
these cover the variants, both halves of split execution (Appendix A,
Algorithm 1), the standalone consensus distance and the access-pattern
reference.  Arrays are filled with a sentinel so that any write shows.
"""

import pytest

from tests import _parity as pa

pytestmark = pytest.mark.gpu

G, ID = ("global",), ("identity",)
RING_MH = ("ring", "metropolis", 0.1)
REG4 = ("regular", "metropolis", 4)
LD = 16  # the row stride of an empty vector still has to keep rows 16-byte aligned


@pytest.fixture(scope="module")
def env():
    import torch

    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    import paper_2606_22768_amd as fgd

    return fgd, torch


def _rows(torch, M, dtype, value):
    t = {"f32": torch.float32, "bf16": torch.bfloat16}[dtype]
    return torch.full((M, LD), value, dtype=t, device="cuda")


def _engine(fgd, M, dtype, spec1, k1, spec2, k2, **kw):
    eng = fgd.Engine(M, 0, LD, dtype, device=0, **kw)
    eng.set_topology_dict("mix1", pa.topo(spec1, M, k1))
    eng.set_topology_dict("mix2", pa.topo(spec2, M, k2))
    return eng


@pytest.mark.parametrize("M,dtype,spec1,k1,spec2,k2,state,nesterov", [
    (8, "bf16", G, 1, RING_MH, 1, True, True),     # GlobalM1SLocalM2
    (8, "f32", RING_MH, 2, RING_MH, 1, True, False),
    (64, "f32", REG4, 1, REG4, 3, False, False),
    (1, "f32", G, 1, ID, 0, True, True),
])
def test_empty_fused_step_variants(env, M, dtype, spec1, k1, spec2, k2, state, nesterov):
    fgd, torch = env
    print(f"[empty] fused M={M} {dtype} state={state} nesterov={nesterov}", flush=True)
    eng = _engine(fgd, M, dtype, spec1, k1, spec2, k2, mix1_state=state, nesterov=nesterov)
    tp, tl, v = _rows(torch, M, dtype, 1.5), _rows(torch, M, dtype, 2.5), _rows(torch, M, "f32", 3.5)
    cd = torch.full((eng.num_cd_rows(), M), 7.0, dtype=torch.float64, device="cuda")
    eng.outer_step(tp, tl, v, cd)
    torch.cuda.synchronize()
    assert torch.all(tp == 1.5) and torch.all(tl == 2.5) and torch.all(v == 3.5)
    assert torch.all(cd == 0)
    eng.close()


@pytest.mark.parametrize("M,dtype,spec1,k1,spec2,k2,state", [
    (8, "bf16", G, 1, RING_MH, 1, False),
    (8, "f32", RING_MH, 2, RING_MH, 1, True),
    (64, "f32", REG4, 1, REG4, 3, False),
])
def test_empty_split_halves(env, M, dtype, spec1, k1, spec2, k2, state):
    fgd, torch = env
    print(f"[empty] split M={M} {dtype} state={state}", flush=True)
    eng = _engine(fgd, M, dtype, spec1, k1, spec2, k2, mix1_state=state)
    n1, n2 = eng.num_cd_rows_split()
    tp, tl, v, x = (_rows(torch, M, dtype, 1.5), _rows(torch, M, dtype, 2.5), _rows(torch, M, "f32", 3.5),
                    _rows(torch, M, dtype, 4.5))
    cd1 = torch.full((n1, M), 7.0, dtype=torch.float64, device="cuda")
    cd2 = torch.full((n2, M), 7.0, dtype=torch.float64, device="cuda")
    eng.mix1(tp, x, v if state else None, cd1)
    eng.outer_step_blocking(x, tp, tl, v, cd2, write_local=True)
    torch.cuda.synchronize()
    assert torch.all(tp == 1.5) and torch.all(tl == 2.5) and torch.all(v == 3.5) and torch.all(x == 4.5)
    assert torch.all(cd1 == 0) and torch.all(cd2 == 0)
    eng.close()


@pytest.mark.parametrize("M,dtype", [(8, "bf16"), (64, "f32"), (3, "f32")])
def test_empty_consensus_distance_and_pattern(env, M, dtype):
    fgd, torch = env
    print(f"[empty] consensus and pattern M={M} {dtype}", flush=True)
    eng = _engine(fgd, M, dtype, G, 1, ID, 0)
    x = _rows(torch, M, dtype, 1.5)
    out = torch.full((M,), 7.0, dtype=torch.float64, device="cuda")
    eng.consensus_distance(x, out)
    torch.cuda.synchronize()
    assert torch.all(out == 0) and torch.all(x == 1.5)
    if M in (1, 2, 4, 8, 16, 32, 64):  # the worker counts the pattern reference is built for
        tl, v = _rows(torch, M, dtype, 2.5), _rows(torch, M, "f32", 3.5)
        eng.stream_step_pattern(x, tl, v)
        torch.cuda.synchronize()
        assert torch.all(x == 1.5) and torch.all(tl == 2.5) and torch.all(v == 3.5)
    eng.close()
