"""GPU parity of prepared operands: curvefp_prepare expands one operand into a buffer of its own
and curvefp_gemm_prepared multiplies two of them.  The expansion depends on the operand alone, so
every case checks the result bit for bit against curvefp_gemm_ws (one format) or
curvefp_gemm_mixed with both operands quantized along K (two formats) on the same codes, and
against the exact phase-binned oracle."""

import numpy as np
import pytest
import torch

import oracle
from paper_2608_10010_amd import curvefp as cf
from paper_2608_10010_amd import workloads as W
from tests.gpu_util import DEV, FMTS, check_gemm, gemm_tolerance, say, to_dev
from tests.test_gpu_gemm import EDGE_PAIRS, oracle_gemm
from tests.test_gpu_gemm_mixed import oracle_mixed
from tests.test_gpu_gemm_ws import same_bits

pytestmark = pytest.mark.gpu


def quantized(X, fmt, dtype="f32", axis=1):
    return cf.curvefp_quantize(to_dev(X, dtype), fmt, block_axis=axis)


def prepared_product(qa, fa, qb, fb, M, N, K, c=None, block=32):
    pa = cf.curvefp_prepare(qa[0], qa[1], M, K, fa, block=block)
    pb = cf.curvefp_prepare(qb[0], qb[1], N, K, fb, block=block)
    return cf.curvefp_gemm_prepared(pa, fa, pb, fb, M, N, K, c=c)


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("shape", [(200, 136, 96), (1, 1, 32), (129, 257, 320), (64, 300, 1024), (300, 520, 640)])
def test_shapes(fmt, shape):
    """Ragged edges, a single element, and K split in two (fewer than 256 output tiles with
    K >= 512: the GEMM's workspace holds the partial sums)."""
    M, N, K = shape
    rng = np.random.default_rng(M * 7 + N + 5 * K)
    A = (rng.standard_normal((M, K)) * np.exp2(rng.uniform(-6, 6, (M, 1)))).astype(np.float32)
    B = (rng.standard_normal((N, K)) * 0.02).astype(np.float32)
    say(f"[gemm_prepared] shapes fmt={fmt} M={M} N={N} K={K}")
    qa, qb = quantized(A, fmt), quantized(B, fmt)
    Cp = prepared_product(qa, fmt, qb, fmt, M, N, K)
    Cw = cf.curvefp_gemm_ws(qa[0], qa[1], qb[0], qb[1], M, N, K, fmt)
    torch.cuda.synchronize()
    Cp, Cw = Cp.cpu().numpy(), Cw.cpu().numpy()
    V, tol = oracle_gemm(A, B, fmt)
    check_gemm(Cp, V, tol, f"prepared {fmt} {shape}")
    same_bits(Cp, Cw, f"prepared {fmt} {shape}")


@pytest.mark.parametrize("fmt", ("E4C3", "E3C3"))
@pytest.mark.parametrize("kind", list(EDGE_PAIRS))
def test_edges(fmt, kind):
    """Zero, poisoned (NaN / infinity), subnormal and wide-range blocks: the prepared buffers carry
    the row maxima, so NaN rows and columns and the scale-spread limit come out as in
    curvefp_gemm_ws."""
    ka, kb = EDGE_PAIRS[kind]
    A = W.edge_tensor(ka, (96, 512), seed=51)
    B = W.edge_tensor(kb, (80, 512), seed=52)
    if kind == "wide_range":
        A = (A * np.float32(2.0 ** -4)).astype(np.float32)
    say(f"[gemm_prepared] edges fmt={fmt} {kind}")
    qa, qb = quantized(A, fmt), quantized(B, fmt)
    Cp = prepared_product(qa, fmt, qb, fmt, 96, 80, 512)
    Cw = cf.curvefp_gemm_ws(qa[0], qa[1], qb[0], qb[1], 96, 80, 512, fmt)
    torch.cuda.synchronize()
    Cp, Cw = Cp.cpu().numpy(), Cw.cpu().numpy()
    V, tol = oracle_gemm(A, B, fmt)
    check_gemm(Cp, V, tol, f"prepared {fmt} {kind}")
    same_bits(Cp, Cw, f"prepared {fmt} {kind}")


@pytest.mark.parametrize("fa", FMTS)
@pytest.mark.parametrize("fb", FMTS)
def test_format_pairs(fa, fb):
    """Two formats: each operand is prepared with its own table and exponent offset, and the GEMM
    removes their sum; the same C as curvefp_gemm_mixed with both operands along K."""
    M, N, K = 136, 264, 384
    rng = np.random.default_rng(7 * FMTS.index(fa) + FMTS.index(fb))
    A = (rng.standard_normal((M, K)) * np.exp2(rng.uniform(-5, 5, (M, 1)))).astype(np.float32)
    B = (rng.standard_normal((N, K)) * np.exp2(rng.uniform(-3, 3, (N, 1)))).astype(np.float32)
    say(f"[gemm_prepared] pair {fa}x{fb} M={M} N={N} K={K}")
    qa, qb = quantized(A, fa), quantized(B, fb)
    Cp = prepared_product(qa, fa, qb, fb, M, N, K)
    Cm = cf.curvefp_gemm_mixed(qa[0], qa[1], fa, 0, qb[0], qb[1], fb, 0, M, N, K)
    torch.cuda.synchronize()
    Cp, Cm = Cp.cpu().numpy(), Cm.cpu().numpy()
    V, tol = oracle_mixed(A, fa, 1, 0, B, fb, 1, 0)
    check_gemm(Cp, V, tol, f"prepared {fa}x{fb}")
    same_bits(Cp, Cm, f"prepared {fa}x{fb}")


def test_prepared_weights_serve_many_products():
    """A weight operand prepared once serves products with activations of several row counts
    (one of them on a second stream), and a larger block size; the prepared buffer is only read."""
    rng = np.random.default_rng(61)
    N, K = 520, 1024
    Wt = (rng.standard_normal((N, K)) * 0.02).astype(np.float32)
    for block in (32, 128):
        qb = cf.curvefp_quantize(to_dev(Wt, "f32"), "E4C3", block=block)
        pb = cf.curvefp_prepare(qb[0], qb[1], N, K, "E4C3", block=block)
        side = torch.cuda.Stream()
        for i, M in enumerate((64, 300, 1100)):
            A = rng.standard_normal((M, K)).astype(np.float32)
            qa = cf.curvefp_quantize(to_dev(A, "f32"), "E4C3", block=block)
            say(f"[gemm_prepared] shared weights block={block} M={M} N={N} K={K}")
            torch.cuda.synchronize()
            if i == 1:
                with torch.cuda.stream(side):
                    pa = cf.curvefp_prepare(qa[0], qa[1], M, K, "E4C3", block=block, stream=side)
                    Cp = cf.curvefp_gemm_prepared(pa, "E4C3", pb, "E4C3", M, N, K, stream=side)
            else:
                pa = cf.curvefp_prepare(qa[0], qa[1], M, K, "E4C3", block=block)
                Cp = cf.curvefp_gemm_prepared(pa, "E4C3", pb, "E4C3", M, N, K)
            Cw = cf.curvefp_gemm_ws(qa[0], qa[1], qb[0], qb[1], M, N, K, "E4C3", block=block)
            torch.cuda.synchronize()
            Cp, Cw = Cp.cpu().numpy(), Cw.cpu().numpy()
            rows = np.arange(0, M, max(1, M // 24))
            f = oracle.get_format("E4C3")
            ca, sa = oracle.quantize(A[rows], f, block)
            cb, sb = oracle.quantize(Wt, f, block)
            V = oracle.gemm_exact(ca, sa, cb, sb, f, block=block)
            tol = gemm_tolerance(ca, sa, cb, sb, "E4C3", block=block)
            check_gemm(Cp[rows], V, tol, f"shared weights block={block} M={M}")
            same_bits(Cp, Cw, f"shared weights block={block} M={M}")


def test_row_stride_and_reused_workspace():
    """An output with a row stride (columns past N untouched), and one workspace for a split-K
    product then a smaller one."""
    rng = np.random.default_rng(71)
    ws = torch.empty(cf.curvefp_gemm_prepared_workspace_bytes(300, 260, 2048), dtype=torch.uint8, device=DEV)
    for (M, N, K) in ((300, 260, 2048), (40, 72, 1024)):
        A = rng.standard_normal((M, K)).astype(np.float32)
        B = rng.standard_normal((N, K)).astype(np.float32)
        qa, qb = quantized(A, "E5C2"), quantized(B, "E5C2")
        say(f"[gemm_prepared] workspace reuse M={M} N={N} K={K}")
        pa = cf.curvefp_prepare(qa[0], qa[1], M, K, "E5C2")
        pb = cf.curvefp_prepare(qb[0], qb[1], N, K, "E5C2")
        out = torch.full((M, N + 12), 5.0, device=DEV)
        cf.curvefp_gemm_prepared(pa, "E5C2", pb, "E5C2", M, N, K, c=out[:, :N], workspace=ws)
        Cw = cf.curvefp_gemm_ws(qa[0], qa[1], qb[0], qb[1], M, N, K, "E5C2")
        torch.cuda.synchronize()
        got, Cw = out.cpu().numpy(), Cw.cpu().numpy()
        V, tol = oracle_gemm(A, B, "E5C2")
        check_gemm(got[:, :N], V, tol, f"prepared ldc {M}x{N}x{K}")
        same_bits(np.ascontiguousarray(got[:, :N]), Cw, f"prepared ldc {M}x{N}x{K}")
        assert np.all(got[:, N:] == 5.0)


@pytest.mark.parametrize("name", ["inference", "dgrad", "sweep_gateup_E4C3", "sweep_down_E3C3", "sweep_qkv_E5C2"])
def test_workload_full_size(name):
    """Full-size products as the benchmark's step runs them (each operand prepared on its own):
    the whole output bit for bit against curvefp_gemm_ws, sampled rows against the oracle."""
    w = W.get(name)
    A, B = w.operand("a"), w.operand("b")
    say(f"[gemm_prepared] workload={name} M={w.M} N={w.N} K={w.K} fmt={w.fmt}")
    qa = quantized(A, w.fmt, w.dtype, w.a.axis)
    qb = quantized(B, w.fmt, w.dtype, w.b.axis)
    Cp = prepared_product(qa, w.fmt, qb, w.fmt, w.M, w.N, w.K)
    Cw = cf.curvefp_gemm_ws(qa[0], qa[1], qb[0], qb[1], w.M, w.N, w.K, w.fmt)
    torch.cuda.synchronize()
    Cp, Cw = Cp.cpu().numpy(), Cw.cpu().numpy()
    rows = np.arange(0, w.M, max(1, w.M // 16))
    cols = np.unique(np.concatenate([np.arange(0, w.N, max(1, w.N // 256)), np.arange(w.N - 32, w.N)]))
    V, tol = oracle_gemm(A, B, w.fmt, w.a.axis, w.b.axis, rows=rows, cols=cols)
    rel = check_gemm(Cp[rows][:, cols], V, tol, name)
    say(f"[gemm_prepared] workload={name} rel_frob={rel:.3e}")
    same_bits(Cp, Cw, name)


# reused forward operands (the backward GEMMs of Sec. 3.3): a [K][R] tensor quantized along R,
# prepared with trans = 1, against curvefp_gemm_mixed with the same layouts
from tests.test_gpu_gemm_mixed import operand_source  # noqa: E402


@pytest.mark.parametrize("fa,fb", [("E5C2", "E4C3"), ("E4C3", "E4C3"), ("E3C3", "E5C2"), ("E4C3_r3/4", "E4C3_r8/9")])
@pytest.mark.parametrize("ta,tb", [(0, 1), (1, 1), (1, 0)])
def test_reused_operands(fa, fb, ta, tb):
    """Each operand prepared in its own layout (ragged M and N, an odd number of K blocks, K not a
    multiple of 256) gives curvefp_gemm_mixed's C bit for bit, within the oracle's bound."""
    M, N, K = 288, 320, 352
    rng = np.random.default_rng(300 + 100 * FMTS.index(fa) + 10 * FMTS.index(fb) + 2 * ta + tb)
    A = operand_source(rng, M, K, ta)
    B = operand_source(rng, N, K, tb, spread=3.0)
    say(f"[gemm_prepared] reused {fa}x{fb} trans={ta}{tb} M={M} N={N} K={K}")
    qa = quantized(A, fa)
    qb = quantized(B, fb)
    pa = cf.curvefp_prepare(qa[0], qa[1], M, K, fa, trans=ta)
    pb = cf.curvefp_prepare(qb[0], qb[1], N, K, fb, trans=tb)
    Cp = cf.curvefp_gemm_prepared(pa, fa, pb, fb, M, N, K)
    Cm = cf.curvefp_gemm_mixed(qa[0], qa[1], fa, ta, qb[0], qb[1], fb, tb, M, N, K)
    torch.cuda.synchronize()
    Cp, Cm = Cp.cpu().numpy(), Cm.cpu().numpy()
    V, tol = oracle_mixed(A, fa, 1, ta, B, fb, 1, tb)
    check_gemm(Cp, V, tol, f"prepared reused {fa}x{fb} trans={ta}{tb}")
    same_bits(Cp, Cm, f"prepared reused {fa}x{fb} trans={ta}{tb}")


@pytest.mark.parametrize("name", ["dgrad_mixed", "wgrad_mixed"])
def test_backward_workload_full_size(name):
    """The 7B up-projection's backward GEMMs as the paper runs them (E5C2 output gradients times
    the reused E4C3 forward codes), every operand prepared: the whole output bit for bit against
    curvefp_gemm_mixed, sampled rows against the oracle."""
    w = W.get(name)
    A, B = w.operand("a"), w.operand("b")
    fa, fb = w.fmt_of("a"), w.fmt_of("b")
    say(f"[gemm_prepared] backward workload={name} M={w.M} N={w.N} K={w.K} {fa}x{fb} "
        f"trans={w.a.trans}{w.b.trans}")
    qa = quantized(A, fa, w.dtype, w.a.axis)
    qb = quantized(B, fb, w.dtype, w.b.axis)
    pa = cf.curvefp_prepare(qa[0], qa[1], w.M, w.K, fa, trans=w.a.trans)
    pb = cf.curvefp_prepare(qb[0], qb[1], w.N, w.K, fb, trans=w.b.trans)
    Cp = cf.curvefp_gemm_prepared(pa, fa, pb, fb, w.M, w.N, w.K)
    Cm = cf.curvefp_gemm_mixed(qa[0], qa[1], fa, w.a.trans, qb[0], qb[1], fb, w.b.trans, w.M, w.N, w.K)
    torch.cuda.synchronize()
    Cp, Cm = Cp.cpu().numpy(), Cm.cpu().numpy()
    same_bits(Cp, Cm, name)
    rows = np.arange(0, w.M, max(1, w.M // 12))
    cols = np.unique(np.concatenate([np.arange(0, w.N, max(1, w.N // 128)), np.arange(w.N - 32, w.N)]))
    V, tol = oracle_mixed(A, fa, w.a.axis, w.a.trans, B, fb, w.b.axis, w.b.trans, rows=rows, cols=cols)
    rel = check_gemm(Cp[rows][:, cols], V, tol, name)
    say(f"[gemm_prepared] backward workload={name} rel_frob={rel:.3e}")
