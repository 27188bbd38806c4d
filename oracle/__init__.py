"""CPU oracle for CurveFP block quantization, dequantization and the CurveFP GEMM.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import, call, link
or execute anything in this package: only ``tests/``, ``__graft_entry__.smoke()``
and the ``cpu_baseline`` leg of ``bench.py`` use it.  It shares no code,
header, table or constant generator with the HIP library; the two meet only in
the seeded input generators (``paper_2608_10010_amd.workloads``), which hold
none of the method's arithmetic.

Everything here is written from the paper (arXiv 2608.10010, "CurveFP"):

* formats and levels        -- Sec. 3.1 "A rational-radix datatype family",
                               Eq. (curvefp-value), Tab. (curvefp-formats)
* block quantizer Q(X)      -- Sec. 3.1 (nearest magnitude in absolute error,
                               saturation at the endpoints, ceil-absmax scale)
* closed product + phases   -- Sec. 3.2, Eq. (curve-index-product),
                               Eq. (phase-count), Eq. (binned-accumulation),
                               App. A.1 (bin addressing)
* storage rate              -- Sec. 3.3, Eq. (effective-rate)

Readings of points the paper leaves open are stated at the function that takes
them.
"""

from .formats import FORMATS, Format, get_format, rational_format
from .quant import (
    scale_exponents,
    quantize,
    quantize_axis0,
    quantize_mse,
    mse_candidates,
    quantize_mse_axis0,
    block_sq_error,
    dequantize,
    code_fields,
    level_value_f64,
    pack7,
    unpack7,
    quantize_compact,
    quantize_tensorwise,
    compact_scales,
    pack_offsets,
    unpack_offsets,
    POISON_SCALE,
)
from .gemm import (
    gemm_exact,
    gemm_exact_mixed,
    mixed_lattice,
    expand_scales,
    product_address_mixed,
    gemm_exact_python,
    product_address,
    phase_bins_one,
    load_library,
)

__all__ = [
    "FORMATS", "Format", "get_format", "rational_format",
    "scale_exponents", "quantize", "quantize_axis0", "quantize_mse", "quantize_mse_axis0", "mse_candidates",
    "block_sq_error", "dequantize",
    "code_fields", "level_value_f64", "pack7", "unpack7", "POISON_SCALE",
    "gemm_exact", "gemm_exact_mixed", "mixed_lattice", "expand_scales", "product_address_mixed",
    "gemm_exact_python", "product_address", "phase_bins_one",
    "load_library",
]
