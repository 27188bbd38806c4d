"""GPU edge cases at the limits of the index arithmetic: a row quantization and a
dequantization whose chunk count passes one launch's 32-bit range (the launches are cut
into slabs), a GEMM with K = 2^20, and outputs whose row stride exceeds 2^20 floats
(the GEMM epilogue then takes its 64-bit addressing path, with and without a K split).
Outputs are checked against the oracle on sampled rows; the largest case needs about
90 GB of device memory and is skipped when that is not free."""

import numpy as np
import pytest
import torch

import oracle
from paper_2608_10010_amd import curvefp as cf
from tests.gpu_util import DEV, check_gemm, layout_codes, oracle_quantize, say, to_dev
from tests.test_gpu_gemm import oracle_gemm

pytestmark = pytest.mark.gpu


def test_slab_boundary_rows_quantize_dequantize():
    R, C = (1 << 29) + 64, 32            # 2^31 + 256 chunks of 8 codes
    need = R * C * (2 + 1 + 4) + R
    free, _ = torch.cuda.mem_get_info()
    if free < need * 1.15:
        pytest.skip(f"needs {need / 2**30:.0f} GiB of free device memory, {free / 2**30:.0f} GiB free")
    say(f"[large] rows={R} cols={C} bf16 -> E4C3 and back")
    g = torch.Generator(device=DEV)
    g.manual_seed(5)
    x = torch.randn((R, C), generator=g, device=DEV, dtype=torch.bfloat16)
    x[R - 1] = 1000.0                    # the very last block, recognizable
    codes, scales = cf.curvefp_quantize(x, "E4C3")
    torch.cuda.synchronize()
    rows = np.array([0, 1, (1 << 29) - 2, (1 << 29) - 1, 1 << 29, (1 << 29) + 1, R - 2, R - 1])
    src = x[torch.from_numpy(rows).to(DEV)].float().cpu().numpy()
    del x
    oc, os_ = oracle_quantize(src, "E4C3", 1)
    got_c = codes[torch.from_numpy(rows).to(DEV)].cpu().numpy()
    got_s = scales[torch.from_numpy(rows).to(DEV)].cpu().numpy()
    assert np.array_equal(got_s, os_)
    assert np.array_equal(got_c, layout_codes(oc, "E4C3").reshape(got_c.shape))
    say("[large] dequantize")
    out = cf.curvefp_dequantize(codes, scales, "E4C3", R, C)
    torch.cuda.synchronize()
    got = out[torch.from_numpy(rows).to(DEV)].cpu().numpy()
    del out, codes, scales
    exp = oracle.dequantize(oc, os_, oracle.get_format("E4C3"))
    assert np.array_equal(got.view(np.uint32), exp.view(np.uint32))


def test_gemm_long_k():
    M, N, K = 64, 64, 1 << 20
    rng = np.random.default_rng(9)
    A = rng.standard_normal((M, K), dtype=np.float32)
    B = rng.standard_normal((N, K), dtype=np.float32)
    say(f"[large] gemm M={M} N={N} K={K}")
    qa = cf.curvefp_quantize(to_dev(A, "f32"), "E5C2")
    qb = cf.curvefp_quantize(to_dev(B, "f32"), "E5C2")
    Cf = cf.curvefp_gemm(qa[0], qa[1], qb[0], qb[1], M, N, K, "E5C2").cpu().numpy()
    Cw = cf.curvefp_gemm_ws(qa[0], qa[1], qb[0], qb[1], M, N, K, "E5C2").cpu().numpy()
    assert np.array_equal(Cf.view(np.uint32), Cw.view(np.uint32))
    rows, cols = np.array([0, 37, 63]), np.array([0, 5, 62, 63])
    V, tol = oracle_gemm(A, B, "E5C2", rows=rows, cols=cols)
    # 2^20 random-sign products: fp32 accumulation error relative to |C| is ~2e-5 here, inside
    # the element-wise bound; the 1e-5 Frobenius bar is for the workloads' K <= 14336
    rel = check_gemm(Cf[rows][:, cols], V, tol, "K = 2^20", frobenius=False)
    say(f"[large] K = 2^20 relative Frobenius error {rel:.2e}")


@pytest.mark.parametrize("K", [64, 1024])    # 1024: the K split, whose halves add with atomics
def test_gemm_very_wide_row_stride(K):
    M, N = 8, 40
    ldc = (1 << 20) + 64
    rng = np.random.default_rng(K)
    A = rng.standard_normal((M, K)).astype(np.float32)
    B = rng.standard_normal((N, K)).astype(np.float32)
    say(f"[large] gemm ldc={ldc} K={K}")
    qa = cf.curvefp_quantize(to_dev(A, "f32"), "E4C3")
    qb = cf.curvefp_quantize(to_dev(B, "f32"), "E4C3")
    V, tol = oracle_gemm(A, B, "E4C3")
    for ws in (False, True):
        out = torch.full((M, ldc), 3.0, device=DEV)
        if ws:
            cf.curvefp_gemm_ws(qa[0], qa[1], qb[0], qb[1], M, N, K, "E4C3", c=out[:, :N])
        else:
            cf.curvefp_gemm(qa[0], qa[1], qb[0], qb[1], M, N, K, "E4C3", c=out[:, :N])
        torch.cuda.synchronize()
        got = out[:, : N + 64].cpu().numpy()
        check_gemm(got[:, :N], V, tol, f"ldc {ldc} ws={ws}")
        assert np.all(got[:, N:] == 3.0)
        assert float(out[:, N + 64:].max()) == 3.0 and float(out[:, N + 64:].min()) == 3.0
