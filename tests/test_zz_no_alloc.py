"""curvefp_gemm_ws_static: the workspace GEMM on the library's static device scratch, for callers
that cannot allocate.  Called through the C ABI (ctypes, raw pointers) and checked against
curvefp_gemm_ws with a caller-allocated workspace (bit for bit: same kernels, same values) and
against the oracle's exact phase-binned sum (the GEMM parity bound), on two calls in a row, the
second smaller than the first and in another format, so it runs on what the first left in the
scratch.  Oversized products are refused before any HIP call."""

import ctypes

import numpy as np
import pytest
import torch

from paper_2608_10010_amd import curvefp as cf
from tests.gpu_util import DEV, check_gemm, say, to_dev
from tests.test_gpu_gemm import oracle_gemm

ESHAPE = -2
STATIC_BYTES = 128 << 20


def static_call(qa, qb, M, N, K, fmt, c):
    L = cf.lib()
    stream = torch.cuda.current_stream()
    return L.curvefp_gemm_ws_static(qa[0].data_ptr(), qa[1].data_ptr(), qb[0].data_ptr(), qb[1].data_ptr(),
                                    M, N, K, cf.FORMATS[fmt], 32, c.data_ptr(), c.stride(0),
                                    ctypes.c_void_p(stream.cuda_stream))


@pytest.mark.gpu
def test_static_scratch_matches_workspace_gemm():
    rng = np.random.default_rng(91)
    cases = [(1536, 1280, 2048, "E4C3"), (200, 136, 320, "E3C3")]
    for M, N, K, fmt in cases:
        assert cf.curvefp_gemm_workspace_bytes(M, N, K) <= STATIC_BYTES
        A = (rng.standard_normal((M, K)) * np.exp2(rng.uniform(-4, 4, (M, 1)))).astype(np.float32)
        B = (rng.standard_normal((N, K)) * 0.02).astype(np.float32)
        say(f"[no_alloc] curvefp_gemm_ws_static M={M} N={N} K={K} fmt={fmt}")
        qa = cf.curvefp_quantize(to_dev(A, "f32"), fmt)
        qb = cf.curvefp_quantize(to_dev(B, "f32"), fmt)
        c = torch.full((M, N), float("nan"), dtype=torch.float32, device=DEV)
        assert static_call(qa, qb, M, N, K, fmt, c) == 0
        ref = cf.curvefp_gemm_ws(qa[0], qa[1], qb[0], qb[1], M, N, K, fmt)
        torch.cuda.synchronize()
        got, want = c.cpu().numpy(), ref.cpu().numpy()
        assert np.array_equal(got.view(np.uint32), want.view(np.uint32)), f"{fmt} {M}x{N}x{K}: differs from ws"
        rows = np.arange(0, M, max(1, M // 64))
        V, tol = oracle_gemm(A, B, fmt, rows=rows)
        rel = check_gemm(got[rows].astype(np.float64), V, tol, f"static {fmt} {M}x{N}x{K}")
        say(f"[no_alloc] {fmt} {M}x{N}x{K} bit-exact with curvefp_gemm_ws, rel_frob={rel:.3e}")


def test_oversized_product_is_refused():
    """Validation runs before any HIP call, so this needs no GPU: a product whose workspace
    exceeds the static scratch returns CURVEFP_ERR_SHAPE."""
    M, N, K = 4096, 4096, 4096
    assert cf.curvefp_gemm_workspace_bytes(M, N, K) > STATIC_BYTES
    p = ctypes.c_void_p(256)            # never dereferenced: the call stops at validation
    st = cf.lib().curvefp_gemm_ws_static(p, p, p, p, M, N, K, 0, 32, p, N, None)
    assert st == ESHAPE
