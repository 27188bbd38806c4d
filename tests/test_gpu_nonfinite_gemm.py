"""GPU parity of the GEMMs on sources that hold NaN or infinity.

Such a value poisons its block (scale -128, zero codes), which reconstructs to NaN, and each
GEMM computes deq(A) deq(B)^T in IEEE terms: every output in a row of A or of B that holds a
poisoned block is NaN (zero partners included), every other output is the usual product.
Checked against the oracle (NaN at exactly its places, the element-wise bound elsewhere) for the
fused, workspace, mixed-format and requantizing entry points, with and without the K split."""

import numpy as np
import pytest
import torch

from paper_2608_10010_amd import curvefp as cf
from tests.gpu_util import BINARY_FMTS, check_gemm, say, to_dev
from tests.test_gpu_gemm import oracle_gemm
from tests.test_gpu_gemm_mixed import gpu_mixed, oracle_mixed

pytestmark = pytest.mark.gpu


def sources(M, N, K, seed):
    rng = np.random.default_rng(seed)
    A = rng.standard_normal((M, K)).astype(np.float32)
    B = (rng.standard_normal((N, K)) * 0.02).astype(np.float32)
    A[3, 5] = np.nan
    A[M - 1, K - 2] = np.inf
    A[M // 2, 40] = -np.inf
    B[2, K // 2] = np.inf
    B[N - 5, 0] = np.nan
    B[7, :32] = 0.0
    B[7, 33] = -np.inf                 # a poisoned block next to an all-zero one
    return A, B


@pytest.mark.parametrize("fmt", BINARY_FMTS + ("E4C3_r3/4",))
@pytest.mark.parametrize("K", [256, 1024])      # 1024: few tiles and 32 blocks, so K is split
def test_fused_and_workspace(fmt, K):
    M, N = 200, 136
    A, B = sources(M, N, K, 61 + K)
    say(f"[nonfinite] fused and ws fmt={fmt} M={M} N={N} K={K}")
    qa = cf.curvefp_quantize(to_dev(A, "f32"), fmt)
    qb = cf.curvefp_quantize(to_dev(B, "f32"), fmt)
    Cf = cf.curvefp_gemm(qa[0], qa[1], qb[0], qb[1], M, N, K, fmt)
    Cw = cf.curvefp_gemm_ws(qa[0], qa[1], qb[0], qb[1], M, N, K, fmt)
    torch.cuda.synchronize()
    Cf, Cw = Cf.cpu().numpy(), Cw.cpu().numpy()
    V, tol = oracle_gemm(A, B, fmt)
    assert np.isnan(V).all(axis=1).sum() == 3 and np.isnan(V).all(axis=0).sum() == 3
    check_gemm(Cf, V, tol, f"fused nonfinite {fmt} K={K}")
    check_gemm(Cw, V, tol, f"ws nonfinite {fmt} K={K}")
    assert np.array_equal(Cf.view(np.uint32), Cw.view(np.uint32))


@pytest.mark.parametrize("ta,tb", [(0, 0), (0, 1), (1, 1)])
def test_mixed(ta, tb):
    """E5C2 x E4C3; a reused operand (trans) holds the codes of its [K][R] transpose, blocks along
    R: a poisoned block there covers 32 GEMM rows of one k."""
    M, N, K = 192, 160, 256
    A, B = sources(M, N, K, 67)
    Ax = np.ascontiguousarray(A.T) if ta else A
    Bx = np.ascontiguousarray(B.T) if tb else B
    say(f"[nonfinite] mixed ta={ta} tb={tb}")
    C = gpu_mixed(Ax, "E5C2", 1, ta, Bx, "E4C3", 1, tb)
    V, tol = oracle_mixed(Ax, "E5C2", 1, ta, Bx, "E4C3", 1, tb)
    assert np.isnan(V).any()
    check_gemm(C, V, tol, f"mixed nonfinite ta={ta} tb={tb}")


@pytest.mark.parametrize("K", [256, 1024])
def test_requant(K):
    """Requantized output equals curvefp_quantize of the fp32 C: the NaN outputs poison their
    output blocks (scale -128, zero codes)."""
    M, N, fmt = 200, 192, "E4C3"
    A, B = sources(M, N, K, 71 + K)
    say(f"[nonfinite] requant K={K}")
    qa = cf.curvefp_quantize(to_dev(A, "f32"), fmt)
    qb = cf.curvefp_quantize(to_dev(B, "f32"), fmt)
    C = cf.curvefp_gemm_ws(qa[0], qa[1], qb[0], qb[1], M, N, K, fmt)
    oc, os_ = cf.curvefp_gemm_requant(qa[0], qa[1], qb[0], qb[1], M, N, K, fmt, "E3C3")
    rc, rs = cf.curvefp_quantize(C, "E3C3")
    torch.cuda.synchronize()
    assert np.array_equal(oc.cpu().numpy(), rc.cpu().numpy())
    assert np.array_equal(os_.cpu().numpy(), rs.cpu().numpy())
    s = os_.cpu().numpy()
    # the three poisoned rows of A poison every output block of their rows; B's poisoned rows
    # (columns 2, 7 and N - 5 of C) poison the output blocks holding those columns in every row
    assert np.all(s[[3, M // 2, M - 1]] == -128)
    col_blocks = sorted({2 // 32, 7 // 32, (N - 5) // 32})
    others = np.setdiff1d(np.arange(M), [3, M // 2, M - 1])
    assert np.all(s[others][:, col_blocks] == -128)
    assert not np.any(s[others][:, np.setdiff1d(np.arange(N // 32), col_blocks)] == -128)
