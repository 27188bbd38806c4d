"""GPU parity of the workspace GEMM (curvefp_gemm_ws): the codes are expanded once into a
workspace and the GEMM streams the expanded planes.  Every case checks the result against the
exact phase-binned oracle (same bound as the fused entry point) and, since the expanded values
and the MFMA order are the same, bit for bit against curvefp_gemm on the same codes."""

import numpy as np
import pytest
import torch

from paper_2608_10010_amd import curvefp as cf
from paper_2608_10010_amd import workloads as W
from tests.gpu_util import DEV, FMTS, check_gemm, say, to_dev
from tests.test_gpu_gemm import EDGE_PAIRS, oracle_gemm

pytestmark = pytest.mark.gpu


def both(A, B, fmt, dtype, a_axis=1, b_axis=1, ws=None):
    qa = cf.curvefp_quantize(to_dev(A, dtype), fmt, block_axis=a_axis)
    qb = cf.curvefp_quantize(to_dev(B, dtype), fmt, block_axis=b_axis)
    M, N, K = qa[1].shape[0], qb[1].shape[0], qa[1].shape[1] * 32
    Cf = cf.curvefp_gemm(qa[0], qa[1], qb[0], qb[1], M, N, K, fmt)
    Cw = cf.curvefp_gemm_ws(qa[0], qa[1], qb[0], qb[1], M, N, K, fmt, workspace=ws)
    torch.cuda.synchronize()
    return Cw.cpu().numpy(), Cf.cpu().numpy()


def same_bits(x, y, what):
    assert x.shape == y.shape
    bad = x.view(np.uint32) != y.view(np.uint32)
    assert not bad.any(), f"{what}: {bad.sum()} elements differ from curvefp_gemm"


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("shape", [(200, 136, 96), (128, 128, 32), (1, 1, 32), (129, 257, 320), (64, 300, 1024),
                                   (300, 520, 640)])
def test_shapes(fmt, shape):
    M, N, K = shape
    rng = np.random.default_rng(M * 5 + N + 3 * K)
    A = (rng.standard_normal((M, K)) * np.exp2(rng.uniform(-6, 6, (M, 1)))).astype(np.float32)
    B = (rng.standard_normal((N, K)) * 0.02).astype(np.float32)
    say(f"[gemm_ws] shapes fmt={fmt} M={M} N={N} K={K}")
    Cw, Cf = both(A, B, fmt, "f32")
    V, tol = oracle_gemm(A, B, fmt)
    check_gemm(Cw, V, tol, f"ws {fmt} {shape}")
    same_bits(Cw, Cf, f"ws {fmt} {shape}")


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("kind", list(EDGE_PAIRS))
def test_edges(fmt, kind):
    ka, kb = EDGE_PAIRS[kind]
    A = W.edge_tensor(ka, (96, 512), seed=31)
    B = W.edge_tensor(kb, (80, 512), seed=32)
    if kind == "wide_range":
        A = (A * np.float32(2.0 ** -4)).astype(np.float32)
    say(f"[gemm_ws] edges fmt={fmt} {kind}")
    Cw, Cf = both(A, B, fmt, "f32")
    V, tol = oracle_gemm(A, B, fmt)
    check_gemm(Cw, V, tol, f"ws {fmt} {kind}")
    same_bits(Cw, Cf, f"ws {fmt} {kind}")


def test_workspace_reuse_and_row_stride():
    """One workspace for a larger then a smaller product (the second must not see the first's
    planes), and an output with a row stride."""
    rng = np.random.default_rng(41)
    ws = cf.gemm_workspace(520, 600, 1024, DEV)
    for (M, N, K) in ((520, 600, 1024), (70, 90, 160)):
        A = rng.standard_normal((M, K)).astype(np.float32)
        B = rng.standard_normal((N, K)).astype(np.float32)
        say(f"[gemm_ws] reuse M={M} N={N} K={K}")
        Cw, Cf = both(A, B, "E5C2", "f32", ws=ws)
        V, tol = oracle_gemm(A, B, "E5C2")
        check_gemm(Cw, V, tol, f"reuse {M}x{N}x{K}")
        same_bits(Cw, Cf, f"reuse {M}x{N}x{K}")
    A = rng.standard_normal((64, 128)).astype(np.float32)
    B = rng.standard_normal((40, 128)).astype(np.float32)
    qa = cf.curvefp_quantize(to_dev(A, "f32"), "E4C3")
    qb = cf.curvefp_quantize(to_dev(B, "f32"), "E4C3")
    out = torch.full((64, 52), 5.0, device=DEV)
    cf.curvefp_gemm_ws(qa[0], qa[1], qb[0], qb[1], 64, 40, 128, "E4C3", c=out[:, :40], workspace=ws)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    V, tol = oracle_gemm(A, B, "E4C3")
    check_gemm(got[:, :40], V, tol, "ws ldc")
    assert np.all(got[:, 40:] == 5.0)


# every configuration the benchmark runs: the inference GEMM, the 7B forward / dgrad / wgrad, and
# the 8B layer sweep (QKV, O, gate/up, down) in each of the three formats
SWEEPS = [f"sweep_{layer}_{fmt}" for layer in ("qkv", "o", "gateup", "down") for fmt in ("E4C3", "E5C2", "E3C3")]
WL = ["inference", "fwd", "dgrad", "wgrad"] + SWEEPS


@pytest.mark.parametrize("name", WL)
def test_workload_full_size(name):
    """Full-size product of each workload as the benchmark launches it: the whole output bit for
    bit against curvefp_gemm, sampled rows against the oracle."""
    w = W.get(name)
    A, B = w.operand("a"), w.operand("b")
    say(f"[gemm_ws] workload={name} M={w.M} N={w.N} K={w.K} fmt={w.fmt}")
    Cw, Cf = both(A, B, w.fmt, w.dtype, w.a.axis, w.b.axis)
    rows = np.arange(0, w.M, max(1, w.M // 16))
    cols = np.unique(np.concatenate([np.arange(0, w.N, max(1, w.N // 256)), np.arange(w.N - 32, w.N)]))
    V, tol = oracle_gemm(A, B, w.fmt, w.a.axis, w.b.axis, rows=rows, cols=cols)
    rel = check_gemm(Cw[rows][:, cols], V, tol, name)
    say(f"[gemm_ws] workload={name} rel_frob={rel:.3e}")
    same_bits(Cw, Cf, name)


@pytest.mark.parametrize("shape", [(4352, 4096, 1024), (4300, 4000, 1056), (8192, 2304, 2048)])
def test_partial_last_round(shape):
    """More tiles than compute units with a partial last round (272, 272 and 288 tiles of
    256 x 256; ragged edges and an odd K-block count in the second).  Rows are sampled across
    every tile row, columns across every tile column and the ragged edge."""
    M, N, K = shape
    rng = np.random.default_rng(M + N + K)
    A = (rng.standard_normal((M, K)) * np.exp2(rng.uniform(-4, 4, (M, 1)))).astype(np.float32)
    B = (rng.standard_normal((N, K)) * 0.02).astype(np.float32)
    say(f"[gemm_ws] partial last round M={M} N={N} K={K}")
    Cw, Cf = both(A, B, "E4C3", "f32")
    rows = np.unique(np.concatenate([np.arange(0, M, 37), np.arange(M - 8, M)]))
    cols = np.unique(np.concatenate([np.arange(0, N, 29), np.arange(N - 8, N)]))
    V, tol = oracle_gemm(A, B, "E4C3", rows=rows, cols=cols)
    rel = check_gemm(Cw[rows][:, cols], V, tol, f"partial last round {shape}")
    same_bits(Cw, Cf, f"partial last round {shape}")
    say(f"[gemm_ws] partial last round rel_frob={rel:.3e}")
