"""GPU parity: curvefp_gemm against the oracle's exact phase-binned GEMM.

Bar: element-wise |C - V| <= 1e-5 sum_k |a_ik b_jk| + 2^-30 (flush term), and
relative Frobenius error <= 1e-5 (see tests/gpu_util.gemm_tolerance)."""

import numpy as np
import pytest
import torch

import oracle
from paper_2608_10010_amd import curvefp as cf
from paper_2608_10010_amd import workloads as W
from tests.gpu_util import (DEV, FMTS, check_gemm, exact_values, gemm_tolerance, layout_codes,
                            oracle_quantize, row_tops, say, to_dev)

pytestmark = pytest.mark.gpu


def gpu_gemm_from_sources(A, B, fmt, dtype, a_axis=1, b_axis=1):
    qa = cf.curvefp_quantize(to_dev(A, dtype), fmt, block_axis=a_axis)
    qb = cf.curvefp_quantize(to_dev(B, dtype), fmt, block_axis=b_axis)
    M = qa[1].shape[0]
    N = qb[1].shape[0]
    K = qa[1].shape[1] * 32
    C = cf.curvefp_gemm(qa[0], qa[1], qb[0], qb[1], M, N, K, fmt)
    torch.cuda.synchronize()
    return C.cpu().numpy(), qa, qb


def _operand_rows(X, axis, idx):
    """The GEMM rows idx of an operand stored with K along axis 1 (or along axis 0)."""
    if idx is None:
        return X, axis
    return (np.ascontiguousarray(X[idx]), 1) if axis == 1 else (np.ascontiguousarray(X[:, idx]), 0)


def oracle_gemm(A, B, fmt, a_axis=1, b_axis=1, rows=None, cols=None):
    A2, ax = _operand_rows(A, a_axis, rows)
    B2, bx = _operand_rows(B, b_axis, cols)
    ca, sa = oracle_quantize(A2, fmt, ax)
    cb, sb = oracle_quantize(B2, fmt, bx)
    f = oracle.get_format(fmt)
    V = oracle.gemm_exact(ca, sa, cb, sb, f)
    return V, gemm_tolerance(ca, sa, cb, sb, fmt)


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("shape", [(200, 136, 96), (128, 128, 32), (1, 1, 32), (129, 257, 320), (64, 300, 1024)])
def test_shapes(fmt, shape):
    M, N, K = shape
    rng = np.random.default_rng(M * 7 + N + K)
    A = (rng.standard_normal((M, K)) * np.exp2(rng.uniform(-6, 6, (M, 1)))).astype(np.float32)
    B = (rng.standard_normal((N, K)) * 0.02).astype(np.float32)
    say(f"[gemm] shapes fmt={fmt} M={M} N={N} K={K}")
    C, _, _ = gpu_gemm_from_sources(A, B, fmt, "f32")
    V, tol = oracle_gemm(A, B, fmt)
    check_gemm(C, V, tol, f"{fmt} {shape}")


EDGE_PAIRS = {
    "constant": ("constant", "constant"),
    "block_spread": ("block_spread", "block_spread"),
    "wide_range": ("wide_range", "one_hot"),       # A scaled by 2^-4 below: no fp32 overflow
    "zeros": ("zeros", "block_spread"),
    "one_hot": ("one_hot", "one_hot"),
    "tiny_x_huge": ("tiny_blocks", "huge_blocks"),
    "huge_x_tiny": ("huge_blocks", "tiny_blocks"),
}


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("kind", list(EDGE_PAIRS))
def test_edges(fmt, kind):
    ka, kb = EDGE_PAIRS[kind]
    A = W.edge_tensor(ka, (96, 256), seed=21)
    B = W.edge_tensor(kb, (80, 256), seed=22)
    if kind == "wide_range":
        A = (A * np.float32(2.0 ** -4)).astype(np.float32)
    say(f"[gemm] edge fmt={fmt} kind={kind}")
    C, _, _ = gpu_gemm_from_sources(A, B, fmt, "f32")
    V, tol = oracle_gemm(A, B, fmt)
    assert np.all(np.isfinite(V)) and np.all(np.abs(V) < 3e38)
    check_gemm(C, V, tol, f"{fmt} {kind}")


@pytest.mark.parametrize("fmt", FMTS)
def test_all_pairwise_products(fmt):
    """C[i, j] is the single product of code i and code j (K = 32, one block):
    every product of the codebook, both signs and zero, through the real kernel."""
    f = oracle.get_format(fmt)
    n = 2 ** (f.E + f.C + 1)
    codes = np.zeros((n, 32), np.uint8)
    codes[:, 0] = np.arange(n)
    sa = np.zeros((n, 1), np.int8)
    rng = np.random.default_rng(23)
    sb = rng.integers(-40, 40, (n, 1)).astype(np.int8)
    say(f"[gemm] all pairwise products fmt={fmt} n={n}")
    ca_d = torch.from_numpy(np.ascontiguousarray(layout_codes(codes, fmt))).to(DEV)
    s_a = torch.from_numpy(sa).to(DEV)
    s_b = torch.from_numpy(sb).to(DEV)
    C = cf.curvefp_gemm(ca_d, s_a, ca_d, s_b, n, n, 32, fmt)
    torch.cuda.synchronize()
    C = C.cpu().numpy().astype(np.float64)
    V = oracle.gemm_exact(codes, sa, codes, sb, f)
    tol = gemm_tolerance(codes, sa, codes, sb, fmt)
    check_gemm(C, V, tol, f"pairwise {fmt}")
    # products of two elements within 2^-12 of their rows' tops are good to 2^-19
    va = np.abs(exact_values(codes, sa, fmt))[:, 0]
    vb = np.abs(exact_values(codes, sb, fmt))[:, 0]
    big = (va[:, None] >= 2.0 ** -12 * row_tops(codes, sa, fmt)[:, None]) & \
          (vb[None, :] >= 2.0 ** -12 * row_tops(codes, sb, fmt)[None, :])
    assert big.sum() > n
    rel = np.abs(C[big] - V[big]) / np.abs(V[big])
    assert rel.max() < 2.0 ** -19, rel.max()


@pytest.mark.parametrize("fmt", FMTS)
def test_sign_symmetry_and_determinism(fmt):
    rng = np.random.default_rng(24)
    A = W.bf16_round(rng.standard_normal((160, 512)).astype(np.float32))
    B = W.bf16_round(rng.standard_normal((96, 512)).astype(np.float32))
    say(f"[gemm] sign symmetry fmt={fmt}")
    C1, qa, qb = gpu_gemm_from_sources(A, B, fmt, "bf16")
    C2, _, _ = gpu_gemm_from_sources(A, B, fmt, "bf16")
    assert np.array_equal(C1.view(np.uint32), C2.view(np.uint32))
    # negating A negates every code-domain product exactly; the MFMA fp32 accumulation is
    # deterministic but not bitwise sign-symmetric, so the two results agree to the bound
    Cn, _, _ = gpu_gemm_from_sources(-A, B, fmt, "bf16")
    V, tol = oracle_gemm(A, B, fmt)
    check_gemm(-Cn, V, tol, "negated A")
    assert np.all(np.abs(Cn + C1) <= 2 * tol)


def test_output_row_stride():
    rng = np.random.default_rng(25)
    A = rng.standard_normal((64, 128)).astype(np.float32)
    B = rng.standard_normal((40, 128)).astype(np.float32)
    qa = cf.curvefp_quantize(to_dev(A, "f32"), "E4C3")
    qb = cf.curvefp_quantize(to_dev(B, "f32"), "E4C3")
    out = torch.full((64, 52), 5.0, device=DEV)
    say("[gemm] ldc 52")
    cf.curvefp_gemm(qa[0], qa[1], qb[0], qb[1], 64, 40, 128, "E4C3", c=out[:, :40])
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    V, tol = oracle_gemm(A, B, "E4C3")
    check_gemm(got[:, :40], V, tol, "ldc")
    assert np.all(got[:, 40:] == 5.0)


SWEEPS = [f"sweep_{layer}_{fmt}" for layer in ("qkv", "o", "gateup", "down") for fmt in ("E4C3", "E5C2", "E3C3")]
WL = ["tiny", "inference", "fwd", "dgrad", "wgrad"] + SWEEPS


@pytest.mark.parametrize("name", WL)
def test_workload_full_size_sampled(name):
    """Full-size GEMM of each workload as the benchmark launches it; rows sampled
    for the oracle (all rows for the tiny workload)."""
    w = W.get(name)
    A, B = w.operand("a"), w.operand("b")
    say(f"[gemm] workload={name} M={w.M} N={w.N} K={w.K} fmt={w.fmt}")
    C, _, _ = gpu_gemm_from_sources(A, B, w.fmt, w.dtype, w.a.axis, w.b.axis)
    assert C.shape == (w.M, w.N)
    rows = np.arange(0, w.M, 1 if w.M <= 256 else max(1, w.M // 24))
    cols = None if w.N <= 256 else np.unique(np.concatenate([np.arange(0, w.N, max(1, w.N // 384)),
                                                             np.arange(w.N - 64, w.N)]))
    V, tol = oracle_gemm(A, B, w.fmt, w.a.axis, w.b.axis, rows=rows, cols=cols)
    Cs = C[rows] if cols is None else C[rows][:, cols]
    rel = check_gemm(Cs, V, tol, name)
    say(f"[gemm] workload={name} sampled {V.shape[0]}x{V.shape[1]} rel_frob={rel:.3e}")
