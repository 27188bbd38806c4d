"""GPU parity of curvefp_gemm_requant: curvefp_gemm_ws's product requantized in the GEMM's
epilogue.  The contract is exact: the codes and scales equal curvefp_quantize (blocks of 32 along
the rows) of the fp32 C that curvefp_gemm_ws returns, bit for bit.  Against the oracle, the codes
of the exact sum (rounded to fp32 and quantized by the oracle) agree except where the fp32 C and
the exact value fall on opposite sides of a decision point, which moves a code by one level."""

import numpy as np
import pytest
import torch

import oracle
from paper_2608_10010_amd import curvefp as cf
from paper_2608_10010_amd import workloads as W
from tests.gpu_util import DEV, FMTS, layout_codes, say, to_dev, unpack_dev_codes
from tests.test_gpu_gemm import EDGE_PAIRS

pytestmark = pytest.mark.gpu


def quantized_operands(A, B, fmt, dtype="f32"):
    qa = cf.curvefp_quantize(to_dev(A, dtype), fmt)
    qb = cf.curvefp_quantize(to_dev(B, dtype), fmt)
    return qa, qb


def fused_and_two_step(qa, qb, M, N, K, fmt, ofmt):
    ws = cf.gemm_workspace(M, N, K, DEV)
    codes, scales = cf.curvefp_gemm_requant(qa[0], qa[1], qb[0], qb[1], M, N, K, fmt, ofmt, workspace=ws)
    C = cf.curvefp_gemm_ws(qa[0], qa[1], qb[0], qb[1], M, N, K, fmt, workspace=ws)
    c2, s2 = cf.curvefp_quantize(C, ofmt)
    torch.cuda.synchronize()
    return (codes.cpu().numpy(), scales.cpu().numpy()), (c2.cpu().numpy(), s2.cpu().numpy()), C


def same(x, y, what):
    assert x[1].shape == y[1].shape and np.array_equal(x[1], y[1]), f"{what}: {np.sum(x[1] != y[1])} scales differ"
    assert np.array_equal(x[0].reshape(-1), y[0].reshape(-1)), \
        f"{what}: {np.sum(x[0].reshape(-1) != y[0].reshape(-1))} code bytes differ"


def sources(M, N, K, seed):
    rng = np.random.default_rng(seed)
    A = (rng.standard_normal((M, K)) * np.exp2(rng.uniform(-4, 4, (M, 1)))).astype(np.float32)
    B = (rng.standard_normal((N, K)) * 0.05).astype(np.float32)
    return A, B


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("ofmt", FMTS)
def test_equals_quantized_gemm_ws(fmt, ofmt):
    """Every input format x output format; ragged M, N a multiple of 32 but not of 256, K split."""
    M, N, K = 300, 544, 640
    A, B = sources(M, N, K, 3 * FMTS.index(fmt) + FMTS.index(ofmt))
    say(f"[gemm_requant] {fmt} -> {ofmt} M={M} N={N} K={K}")
    qa, qb = quantized_operands(A, B, fmt)
    fused, ref, _ = fused_and_two_step(qa, qb, M, N, K, fmt, ofmt)
    same(fused, ref, f"{fmt} -> {ofmt}")


@pytest.mark.parametrize("shape", [(4096, 4096, 128), (256, 288, 32), (40, 32, 96)])
def test_shapes(shape):
    """No K split (256 tiles), a single K block, a single partial tile."""
    M, N, K = shape
    A, B = sources(M, N, K, M + N + K)
    say(f"[gemm_requant] shape {shape}")
    qa, qb = quantized_operands(A, B, "E4C3")
    for ofmt in ("E4C3", "E3C3"):
        fused, ref, _ = fused_and_two_step(qa, qb, M, N, K, "E4C3", ofmt)
        same(fused, ref, f"{shape} -> {ofmt}")


@pytest.mark.parametrize("kind", list(EDGE_PAIRS))
def test_edges(kind):
    ka, kb = EDGE_PAIRS[kind]
    A = W.edge_tensor(ka, (96, 256), seed=61)
    B = W.edge_tensor(kb, (64, 256), seed=62)
    if kind == "wide_range":
        A = (A * np.float32(2.0 ** -4)).astype(np.float32)
    say(f"[gemm_requant] edge {kind}")
    qa, qb = quantized_operands(A, B, "E5C2")
    for ofmt in ("E5C2", "E3C3"):
        fused, ref, _ = fused_and_two_step(qa, qb, 96, 64, 256, "E5C2", ofmt)
        same(fused, ref, f"edge {kind} -> {ofmt}")


@pytest.mark.parametrize("ofmt", FMTS)
def test_against_oracle(ofmt):
    """Codes of the oracle's exact sum (rounded to fp32, quantized by the oracle) against the fused
    codes: blocks whose fp32 maxima agree have the same scale, and a code differs only where the
    fp32 C and the exact value straddle a decision point (one level apart)."""
    M, N, K = 128, 256, 512
    A, B = sources(M, N, K, 77)
    f = oracle.get_format("E4C3")
    fo = oracle.get_format(ofmt)
    qa, qb = quantized_operands(A, B, "E4C3")
    fused, _, C = fused_and_two_step(qa, qb, M, N, K, "E4C3", ofmt)
    ca, sa = oracle.quantize(A, f)
    cb, sb = oracle.quantize(B, f)
    V = oracle.gemm_exact(ca, sa, cb, sb, f).astype(np.float32)
    oc, osc = oracle.quantize(V, fo)
    gc = unpack_dev_codes(torch.from_numpy(fused[0]), ofmt, N)
    gs = fused[1]
    say(f"[gemm_requant] oracle {ofmt}: scales differ in {np.sum(gs != osc)} of {gs.size} blocks, "
        f"codes in {np.sum(gc != oc)} of {gc.size}")
    assert np.mean(gs != osc) < 1e-2
    keep = np.repeat(gs == osc, 32, axis=1)
    nz, s, n = oracle.code_fields(gc, fo)
    nz2, s2, n2 = oracle.code_fields(oc, fo)
    ok = (gc == oc) | ((np.abs(np.where(nz, n, fo.n_min - 1) - np.where(nz2, n2, fo.n_min - 1)) <= 1) & (s == s2))
    assert np.all(ok[keep])
    assert np.mean(gc[keep] != oc[keep]) < 1e-3


@pytest.mark.parametrize("ofmt", ["E3C3", "E4C3"])
def test_inference_full_size(ofmt):
    """The inference GEMM (2048 x 4096 x 4096, E3C3 operands from bf16) requantized for the next
    layer, the whole output bit for bit against the two-step route."""
    w = W.get("inference")
    say(f"[gemm_requant] inference full size -> {ofmt}")
    qa, qb = quantized_operands(w.operand("a"), w.operand("b"), w.fmt, w.dtype)
    fused, ref, _ = fused_and_two_step(qa, qb, w.M, w.N, w.K, w.fmt, ofmt)
    same(fused, ref, f"inference -> {ofmt}")


@pytest.mark.parametrize("ofmt", FMTS)
@pytest.mark.parametrize("G,shape", [(64, (300, 576, 640)), (128, (200, 384, 1024)), (256, (130, 768, 512)),
                                     (64, (2048, 4096, 4096)), (256, (4096, 4096, 128))])
def test_output_blocks_of_g(ofmt, G, shape):
    """Output blocks of 64, 128 and 256 (the next layer's activations at the paper's G64): equal
    to curvefp_quantize of curvefp_gemm_ws's fp32 C with that block, bit for bit; ragged M, N a
    multiple of G but not of 256, K split and not, and the full inference shape."""
    M, N, K = shape
    fmt = "E3C3"
    A, B = sources(M, N, K, G + FMTS.index(ofmt))
    say(f"[gemm_requant] out blocks of {G}: {fmt} -> {ofmt} M={M} N={N} K={K}")
    qa, qb = quantized_operands(A, B, fmt)
    ws = cf.gemm_workspace(M, N, K, DEV)
    codes, scales = cf.curvefp_gemm_requant(qa[0], qa[1], qb[0], qb[1], M, N, K, fmt, ofmt, workspace=ws,
                                            out_block=G)
    C = cf.curvefp_gemm_ws(qa[0], qa[1], qb[0], qb[1], M, N, K, fmt, workspace=ws)
    c2, s2 = cf.curvefp_quantize(C, ofmt, block=G)
    torch.cuda.synchronize()
    same((codes.cpu().numpy(), scales.cpu().numpy()), (c2.cpu().numpy(), s2.cpu().numpy()), f"G={G} -> {ofmt}")
