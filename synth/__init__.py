"""Seeded synthetic inputs shared by the tests, the benchmark and smoke().

This package generates graph structures, given mixing weights, edge masks and
parameter/momentum tensors.  It holds none of the outer step's arithmetic: no
mixing, no reweighting, no optimizer update and no consensus distance.  Both the
CPU oracle and the HIP engine receive what is generated here as plain inputs.
"""

from . import configs, graphs, tensors  # noqa: F401
