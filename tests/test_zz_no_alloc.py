"""fgd_consensus_distance_noalloc, the consensus distance for callers that
cannot allocate: through the C ABI it gives the same bits as
fgd_consensus_distance (same grid and summation order) and matches the
oracle's S_m (Sec. 4.4; Appendix D.1), on consecutive calls that share the
library's static scratch, the second on a smaller input."""

import numpy as np
import pytest

import oracle
from synth import tensors
from tests import _parity as pa

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def env():
    import torch

    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    import paper_2606_22768_amd as fgd

    return fgd, torch


def _dev(torch, a, dtype):
    t = torch.from_numpy(np.ascontiguousarray(a.view(np.int16) if dtype == "bf16" else a)).cuda()
    return t.view(torch.bfloat16) if dtype == "bf16" else t


# (M, P, dtype) pairs: the first call, then a smaller one on the same scratch.
CALLS = [
    ((64, 300_007, "f32"), (64, 1_001, "f32")),
    ((8, 1_000_003, "bf16"), (5, 77, "bf16")),
    ((16, 262_144, "f32"), (3, 0, "f32")),
    ((64, 600_000, "bf16"), (1, 9_999, "f32")),
]


@pytest.mark.parametrize("calls", CALLS, ids=lambda c: f"{c[0]}-then-{c[1]}")
def test_noalloc_matches_the_engine_call_and_the_oracle(env, calls):
    fgd, torch = env
    for M, P, dtype in calls:
        print(f"[noalloc] M={M} P={P} {dtype}", flush=True)
        ld = pa.aligned_ld(P)
        tp, _, _ = tensors.numpy_inputs(M, P, ld=ld, dtype=dtype, seed=M + P)
        x = _dev(torch, tp, dtype)
        got = torch.full((M,), float("nan"), dtype=torch.float64, device="cuda")
        fgd.fgd_consensus_distance_noalloc(M, P, ld, dtype, x, got)
        torch.cuda.synchronize()
        eng = fgd.Engine(M, P, ld, dtype, device=0)
        try:
            want = torch.full((M,), float("nan"), dtype=torch.float64, device="cuda")
            eng.consensus_distance(x, want)
            torch.cuda.synchronize()
        finally:
            eng.close()
        g, w = got.cpu().numpy(), want.cpu().numpy()
        assert np.array_equal(g.view(np.uint64), w.view(np.uint64)), (g, w)
        ref = oracle.consensus(tp, P=P, dtype=dtype)
        scale = float(np.abs(tensors.bf16_bits_to_f32(tp) if dtype == "bf16" else tp).max()) if P else 0.0
        pa.compare_cd(g[None, :], np.asarray(ref)[None, :], pa.cd_floor(P, scale))


def test_noalloc_rejects_more_workers_than_the_scratch_holds(env):
    fgd, torch = env
    x = torch.zeros((65, 16), dtype=torch.float32, device="cuda")
    out = torch.zeros(65, dtype=torch.float64, device="cuda")
    with pytest.raises(fgd.FgdError, match="num_workers 65"):
        fgd.fgd_consensus_distance_noalloc(65, 16, 16, "f32", x, out)
