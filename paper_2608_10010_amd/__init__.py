"""CurveFP on MI355X: block quantization into CurveFP8 E4C3/E5C2 and CurveFP7 E3C3
codes, dequantization, and the CurveFP GEMM, as hand-written HIP kernels for
gfx950 behind a C ABI (``include/curvefp.h``).

``paper_2608_10010_amd.curvefp`` is the thin Python binding (argument
marshalling only); ``paper_2608_10010_amd.workloads`` draws seeded inputs.
"""

__all__ = ["curvefp", "workloads"]
