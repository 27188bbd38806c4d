"""GPU parity of curvefp_gemm_mixed: operands of any two formats, each either quantized along K
or a forward operand reused by a backward GEMM (codes of a [K][R] tensor, blocks along R, so
every element has its own scale along k).  The oracle is the exact mixed-format phase-binned
GEMM (indices lifted to the finer curve lattice, per-element scales), on the oracle's own
quantization of the same seeded sources; the bound is gemm_tolerance's, per operand format."""

import numpy as np
import pytest
import torch

import oracle
from paper_2608_10010_amd import curvefp as cf
from paper_2608_10010_amd import workloads as W
from tests.gpu_util import (DEV, FMTS, check_gemm, gemm_tolerance_mixed, layout_codes, oracle_quantize, say,
                            to_dev)
from tests.test_gpu_gemm import EDGE_PAIRS

pytestmark = pytest.mark.gpu


# ---------------------------------------------------------------- oracle side

def oracle_operand(X, fmt, axis, trans, idx=None):
    """Oracle codes [R][K] (one per byte) and per-element scales [R][K] of a GEMM operand whose
    source X is quantized along `axis` into Q; trans = 0: Q is [R][K], trans = 1: Q is [K][R].
    idx selects GEMM rows; a reused operand is quantized over whole blocks of 32 of them."""
    f = oracle.get_format(fmt)
    if not trans:
        if idx is not None:
            X = np.ascontiguousarray(X[idx] if axis == 1 else X[:, idx])
        c, s = oracle_quantize(X, fmt, axis)
        return c, oracle.expand_scales(s, 32, axis=1)
    pos = None
    if idx is not None:
        blocks = np.unique(np.asarray(idx) // 32)
        sel = (32 * blocks[:, None] + np.arange(32)[None, :]).reshape(-1)
        X = np.ascontiguousarray(X[:, sel] if axis == 1 else X[sel])
        pos = np.searchsorted(sel, idx)
    c, s = oracle_quantize(X, fmt, axis)            # Q [K][R'] with blocks along R'
    c = np.ascontiguousarray(c.T)
    s = oracle.expand_scales(s, 32, axis=0)
    if pos is not None:
        c, s = c[pos], s[pos]
    return c, s


def oracle_mixed(A, fa, a_axis, ta, B, fb, b_axis, tb, rows=None, cols=None):
    ca, sa = oracle_operand(A, fa, a_axis, ta, rows)
    cb, sb = oracle_operand(B, fb, b_axis, tb, cols)
    V = oracle.gemm_exact_mixed(ca, sa, oracle.get_format(fa), cb, sb, oracle.get_format(fb))
    return V, gemm_tolerance_mixed(ca, sa, fa, cb, sb, fb)


# ---------------------------------------------------------------- GPU side

def gpu_operand(X, fmt, dtype, axis):
    codes, scales = cf.curvefp_quantize(to_dev(X, dtype), fmt, block_axis=axis)
    return codes, scales


def gpu_mixed(A, fa, a_axis, ta, B, fb, b_axis, tb, dtype="f32", ws=None):
    ca, sa = gpu_operand(A, fa, dtype, a_axis)
    cb, sb = gpu_operand(B, fb, dtype, b_axis)
    # GEMM sizes from the quantized shapes: scales are [rows][blocks of 32]
    M = sa.shape[1] * 32 if ta else sa.shape[0]
    N = sb.shape[1] * 32 if tb else sb.shape[0]
    K = sa.shape[0] if ta else sa.shape[1] * 32
    C = cf.curvefp_gemm_mixed(ca, sa, fa, ta, cb, sb, fb, tb, M, N, K, workspace=ws)
    torch.cuda.synchronize()
    return C.cpu().numpy()


def source(rng, shape, spread=6.0, row_axis=0):
    """N(0,1) with a per-line magnitude 2^U(-spread, spread) along row_axis."""
    x = rng.standard_normal(shape)
    if row_axis == 0:
        x = x * np.exp2(rng.uniform(-spread, spread, (shape[0], 1)))
    else:
        x = x * np.exp2(rng.uniform(-spread, spread, (1, shape[1])))
    return x.astype(np.float32)


def operand_source(rng, R, K, trans, spread=6.0):
    """Source of a GEMM operand with R rows over K: [R][K] (trans 0) or [K][R] (trans 1), with
    magnitudes varying along k, so a reused operand's scales change along its contraction."""
    if trans:
        return source(rng, (K, R), spread, row_axis=0)
    return source(rng, (R, K), spread, row_axis=0)


# ---------------------------------------------------------------- tests

@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("shape", [(200, 136, 96), (300, 520, 640), (1, 1, 32)])
def test_single_format_matches_ws(fmt, shape):
    """Both operands along K in one format: the mixed entry point is curvefp_gemm_ws bit for bit."""
    M, N, K = shape
    rng = np.random.default_rng(M + 3 * N + 7 * K)
    A = source(rng, (M, K))
    B = (rng.standard_normal((N, K)) * 0.02).astype(np.float32)
    say(f"[gemm_mixed] single-format fmt={fmt} M={M} N={N} K={K}")
    ca, sa = gpu_operand(A, fmt, "f32", 1)
    cb, sb = gpu_operand(B, fmt, "f32", 1)
    Cm = cf.curvefp_gemm_mixed(ca, sa, fmt, 0, cb, sb, fmt, 0, M, N, K)
    Cw = cf.curvefp_gemm_ws(ca, sa, cb, sb, M, N, K, fmt)
    torch.cuda.synchronize()
    Cm, Cw = Cm.cpu().numpy(), Cw.cpu().numpy()
    assert np.array_equal(Cm.view(np.uint32), Cw.view(np.uint32)), f"{fmt} {shape}"
    V, tol = oracle_mixed(A, fmt, 1, 0, B, fmt, 1, 0)
    check_gemm(Cm, V, tol, f"single {fmt} {shape}")


PAIRS = [(fa, fb) for fa in FMTS for fb in FMTS]


@pytest.mark.parametrize("fa,fb", PAIRS)
@pytest.mark.parametrize("ta,tb", [(0, 0), (0, 1), (1, 0), (1, 1)])
def test_pairs_and_layouts(fa, fb, ta, tb):
    """Every format pair in every layout combination; two tile rows and columns, ragged edges
    (M, N not multiples of 256), an odd number of K blocks."""
    M, N, K = 288, 320, 352
    rng = np.random.default_rng(100 * FMTS.index(fa) + 10 * FMTS.index(fb) + 2 * ta + tb)
    A = operand_source(rng, M, K, ta)
    B = operand_source(rng, N, K, tb, spread=3.0)
    say(f"[gemm_mixed] pair {fa}x{fb} trans={ta}{tb} M={M} N={N} K={K}")
    C = gpu_mixed(A, fa, 1, ta, B, fb, 1, tb)
    V, tol = oracle_mixed(A, fa, 1, ta, B, fb, 1, tb)
    rel = check_gemm(C, V, tol, f"{fa}x{fb} trans={ta}{tb}")
    say(f"[gemm_mixed] pair {fa}x{fb} trans={ta}{tb} rel_frob={rel:.3e}")


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("which", ["a", "b"])
def test_reused_layout_equals_k_layout(fmt, which):
    """The same values presented both ways give the same C bit for bit: codes with scales that are
    constant on 32 x 32 tiles are at once blocked along K ([R][K] codes, scales [R][K/32]) and
    along R ([K][R] codes, scales [K][R/32]).  Host-made random codes; also against the oracle."""
    R, K, O = 320, 384, 200           # rows of the operand under test, K, rows of the other
    rng = np.random.default_rng(7 + FMTS.index(fmt) + (which == "b"))
    f = oracle.get_format(fmt)
    bits = f.E + f.C + 1
    codes = rng.integers(0, 1 << bits, size=(R, K), dtype=np.int64).astype(np.uint8)
    codes[rng.random((R, K)) < 0.05] = 0
    tiles = rng.integers(-12, 12, size=(R // 32, K // 32)).astype(np.int8)
    tiles[0, 0] = -20                 # a block more than 24 binades below its rows' top
    tiles[1, :] = 0
    tiles[1, 3] = 27
    s_k = np.repeat(tiles, 32, axis=0)                              # [R][K/32]
    s_r = np.ascontiguousarray(np.repeat(tiles.T, 32, axis=0))      # [K][R/32]
    other = oracle.quantize(source(rng, (O, K)), f)                 # the other operand, along K
    dev = lambda x: torch.from_numpy(np.ascontiguousarray(x)).to(DEV)
    ck = dev(layout_codes(codes, fmt))
    cr = dev(layout_codes(np.ascontiguousarray(codes.T), fmt))
    oc, osc = dev(layout_codes(other[0], fmt)), dev(other[1])
    say(f"[gemm_mixed] reused == K layout fmt={fmt} operand={which}")
    if which == "a":
        C0 = cf.curvefp_gemm_mixed(ck, dev(s_k), fmt, 0, oc, osc, fmt, 0, R, O, K)
        C1 = cf.curvefp_gemm_mixed(cr, dev(s_r), fmt, 1, oc, osc, fmt, 0, R, O, K)
    else:
        C0 = cf.curvefp_gemm_mixed(oc, osc, fmt, 0, ck, dev(s_k), fmt, 0, O, R, K)
        C1 = cf.curvefp_gemm_mixed(oc, osc, fmt, 0, cr, dev(s_r), fmt, 1, O, R, K)
    torch.cuda.synchronize()
    C0, C1 = C0.cpu().numpy(), C1.cpu().numpy()
    assert np.array_equal(C0.view(np.uint32), C1.view(np.uint32)), f"{fmt} {which}"
    se = oracle.expand_scales(s_k, 32, axis=1)
    so = oracle.expand_scales(other[1], 32, axis=1)
    if which == "a":
        V = oracle.gemm_exact_mixed(codes, se, f, other[0], so, f)
        tol = gemm_tolerance_mixed(codes, se, fmt, other[0], so, fmt)
    else:
        V = oracle.gemm_exact_mixed(other[0], so, f, codes, se, f)
        tol = gemm_tolerance_mixed(other[0], so, fmt, codes, se, fmt)
    check_gemm(C1, V, tol, f"reused {fmt} {which}")


# Rows whose elements span far more than the expansion's window (about 2^-39 below the row's
# top, where fp16 subnormals end): terms below it are dropped, which the element-wise bound
# covers, but when the dropped terms meet the other operand's largest elements they can carry
# much of |C|, so the relative Frobenius criterion (meant for data within the window) is not
# applied.  With a reused operand each of the 256 k-elements of a row has its own scale, so the
# tiny/huge block draws (40 binades of block scales) reach that case.
WIDE = ("wide_range", "tiny_x_huge", "huge_x_tiny")


@pytest.mark.parametrize("kind", list(EDGE_PAIRS))
@pytest.mark.parametrize("ta,tb", [(0, 1), (1, 1)])
def test_edges(kind, ta, tb):
    """Edge tensors as E5C2 gradients times reused E4C3 operands.  A reused source [K][R] drawn
    with per-block scales along R has a different scale at every k: block_spread puts them over
    +-40 binades, so elements fall below fp16's range relative to their row's top."""
    ka, kb = EDGE_PAIRS[kind]
    M, N, K = 96, 160, 256
    A = W.edge_tensor(ka, (K, M) if ta else (M, K), seed=51)
    B = W.edge_tensor(kb, (K, N) if tb else (N, K), seed=52)
    if kind == "wide_range":
        A = (A * np.float32(2.0 ** -4)).astype(np.float32)
    say(f"[gemm_mixed] edge {kind} E5C2xE4C3 trans={ta}{tb}")
    C = gpu_mixed(A, "E5C2", 1, ta, B, "E4C3", 1, tb)
    V, tol = oracle_mixed(A, "E5C2", 1, ta, B, "E4C3", 1, tb)
    rel = check_gemm(C, V, tol, f"edge {kind} trans={ta}{tb}", frobenius=kind not in WIDE)
    say(f"[gemm_mixed] edge {kind} trans={ta}{tb} rel_frob={rel:.3e}")


def test_workspace_reuse_and_row_stride():
    """One workspace for a larger then a smaller mixed product, and an output with a row stride."""
    rng = np.random.default_rng(77)
    ws = cf.gemm_mixed_workspace(544, 640, 1024, DEV)
    for (M, N, K, ta, tb) in ((544, 640, 1024, 1, 1), (64, 96, 160, 0, 1)):
        A = operand_source(rng, M, K, ta)
        B = operand_source(rng, N, K, tb)
        say(f"[gemm_mixed] reuse M={M} N={N} K={K} trans={ta}{tb}")
        C = gpu_mixed(A, "E5C2", 1, ta, B, "E4C3", 1, tb, ws=ws)
        V, tol = oracle_mixed(A, "E5C2", 1, ta, B, "E4C3", 1, tb)
        check_gemm(C, V, tol, f"reuse {M}x{N}x{K}")
    A = operand_source(rng, 64, 128, 0)
    B = operand_source(rng, 64, 128, 1)
    ca, sa = gpu_operand(A, "E5C2", "f32", 1)
    cb, sb = gpu_operand(B, "E4C3", "f32", 1)
    out = torch.full((64, 80), 5.0, device=DEV)
    cf.curvefp_gemm_mixed(ca, sa, "E5C2", 0, cb, sb, "E4C3", 1, 64, 64, 128, c=out[:, :64], workspace=ws)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    V, tol = oracle_mixed(A, "E5C2", 1, 0, B, "E4C3", 1, 1)
    check_gemm(got[:, :64], V, tol, "mixed ldc")
    assert np.all(got[:, 64:] == 5.0)


@pytest.mark.parametrize("name", ["dgrad_mixed", "wgrad_mixed"])
def test_workload_full_size(name):
    """The backward GEMMs of the 7B up-projection as the paper runs them (E5C2 output gradients
    times the reused E4C3 forward codes), full size, in the launch the benchmark times; sampled
    rows and columns (whole tiles' edges included) against the oracle."""
    w = W.get(name)
    A, B = w.operand("a"), w.operand("b")
    fa, fb = w.fmt_of("a"), w.fmt_of("b")
    say(f"[gemm_mixed] workload={name} M={w.M} N={w.N} K={w.K} {fa}x{fb} trans={w.a.trans}{w.b.trans}")
    C = gpu_mixed(A, fa, w.a.axis, w.a.trans, B, fb, w.b.axis, w.b.trans, dtype=w.dtype)
    rows = np.unique(np.concatenate([np.arange(0, w.M, max(1, w.M // 24)), np.arange(w.M - 4, w.M)]))
    cols = np.unique(np.concatenate([np.arange(0, w.N, max(1, w.N // 256)), np.arange(w.N - 32, w.N)]))
    V, tol = oracle_mixed(A, fa, w.a.axis, w.a.trans, B, fb, w.b.axis, w.b.trans, rows=rows, cols=cols)
    rel = check_gemm(C[rows][:, cols], V, tol, name)
    say(f"[gemm_mixed] workload={name} rel_frob={rel:.3e}")
