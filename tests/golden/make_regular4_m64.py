"""Writes regular4_m64_seed0.json: the seeded random 4-regular structure on 64
workers used by the M=64 workload.  It is an input fixture (a graph), not an
expected value; it is stored so the workload does not depend on numpy's
generator across versions.  Run from the repository root:

    python tests/golden/make_regular4_m64.py
"""
import json
import os
import sys

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__)))))
from synth import graphs  # noqa: E402

rp, ci = graphs.random_regular(64, 4, seed=0)
out = os.path.join(os.path.dirname(os.path.abspath(__file__)), "regular4_m64_seed0.json")
with open(out, "w") as f:
    json.dump({"source": "synth.graphs.random_regular(64, 4, seed=0), configuration model",
               "M": 64, "degree": 4, "row_ptr": rp.tolist(), "col_idx": ci.tolist()}, f)
print(out, len(ci))
