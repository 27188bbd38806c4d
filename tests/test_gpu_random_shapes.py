"""Seeded random shapes through every single-format GEMM entry point: for each case (M, N, K, format,
block size drawn from one generator), curvefp_gemm, curvefp_gemm_ws and prepare + gemm_prepared give
the same C bit for bit, and sampled rows agree with the exact phase-binned oracle within the GEMM
parity bound.  Shapes span single partial tiles, ragged edges, K split in two and several rounds of
tiles; block sizes 32, 64, 128 and rowwise."""

import numpy as np
import pytest
import torch

import oracle
from paper_2608_10010_amd import curvefp as cf
from tests.gpu_util import FMTS, check_gemm, gemm_tolerance, say, to_dev

pytestmark = pytest.mark.gpu


def cases(n=24, seed=20261202):
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n):
        M = int(rng.choice([1, 7, 64, 255, 256, 257, 600, 1100, 2100]))
        N = int(rng.choice([1, 33, 128, 255, 300, 513, 900, 1500]))
        kb = int(rng.choice([1, 2, 3, 5, 16, 17, 40, 64]))       # K in blocks of 32
        block = int(rng.choice([32, 32, 64, 128, 0]))            # 0: rowwise (one scale per row)
        K = 32 * kb
        if block == 0:
            block = K
        elif K % block:
            block = 32
        fmt = FMTS[int(rng.integers(len(FMTS)))]
        out.append((i, M, N, K, fmt, block))
    return out


@pytest.mark.parametrize("case", cases(), ids=lambda c: f"{c[0]}-{c[1]}x{c[2]}x{c[3]}-{c[4]}-G{c[5]}")
def test_random_shape(case):
    i, M, N, K, fmt, block = case
    rng = np.random.default_rng(1000 + i)
    A = (rng.standard_normal((M, K)) * np.exp2(rng.uniform(-8, 8, (M, 1)))).astype(np.float32)
    B = (rng.standard_normal((N, K)) * np.exp2(rng.uniform(-3, 3, (N, 1)))).astype(np.float32)
    say(f"[random] case {i}: M={M} N={N} K={K} fmt={fmt} G={block}")
    qa = cf.curvefp_quantize(to_dev(A, "f32"), fmt, block=block)
    qb = cf.curvefp_quantize(to_dev(B, "f32"), fmt, block=block)
    Cf = cf.curvefp_gemm(qa[0], qa[1], qb[0], qb[1], M, N, K, fmt, block=block)
    Cw = cf.curvefp_gemm_ws(qa[0], qa[1], qb[0], qb[1], M, N, K, fmt, block=block)
    pa = cf.curvefp_prepare(qa[0], qa[1], M, K, fmt, block=block)
    pb = cf.curvefp_prepare(qb[0], qb[1], N, K, fmt, block=block)
    Cp = cf.curvefp_gemm_prepared(pa, fmt, pb, fmt, M, N, K)
    torch.cuda.synchronize()
    Cf, Cw, Cp = Cf.cpu().numpy(), Cw.cpu().numpy(), Cp.cpu().numpy()
    assert np.array_equal(Cw.view(np.uint32), Cf.view(np.uint32)), "workspace vs fused"
    assert np.array_equal(Cp.view(np.uint32), Cf.view(np.uint32)), "prepared vs fused"
    rows = np.unique(np.concatenate([np.arange(0, M, max(1, M // 12)), [M - 1]]))
    f = oracle.get_format(fmt)
    ca, sa = oracle.quantize(A[rows], f, block)
    cb, sb = oracle.quantize(B, f, block)
    V = oracle.gemm_exact(ca, sa, cb, sb, f, block=block)
    rel = check_gemm(Cf[rows], V, gemm_tolerance(ca, sa, cb, sb, fmt, block=block), f"random case {i}")
    say(f"[random] case {i} rel_frob={rel:.3e}")
