"""MI355X-native hot path of "Adaptive Block-Scaled Data Types": the IF4
block quantizer and the IF4 x IF4 GEMM (with NVFP4, IF3 and IF6 variants),
as hand-written HIP kernels for gfx950 behind the C ABI of include/ifq.h.

`ops` is the Python binding (same names as the C entry points);
`workloads` generates the seeded synthetic input tensors.
"""
from . import ops  # noqa: F401

__all__ = ["ops"]
