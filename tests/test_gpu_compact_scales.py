"""GPU parity of S-bit scale exponents (Eq. effective-rate's S; Sec. 4.2 prices E3C3 weights at
S = 4 and activations at S = 5): curvefp_quantize_compact's codes, row references and packed
offsets bit for bit against the oracle's quantize_compact / pack_offsets, curvefp_scales_unpack
against compact_scales, and the operands consumed by dequantize and the workspace GEMM."""

import numpy as np
import pytest
import torch

import oracle
from paper_2608_10010_amd import curvefp as cf
from paper_2608_10010_amd import workloads as W
from tests.gpu_util import FMTS, check_gemm, gemm_tolerance, layout_codes, say, to_dev

pytestmark = pytest.mark.gpu


def spread_rows(rng, rows, cols, G, spread, zero_frac=0.1):
    """Blocks of G with magnitudes 2^U(0, spread) below a row top of 2^U(-5, 5), some all zero."""
    top = rng.uniform(-5, 5, (rows, 1))
    blk = top - rng.uniform(0, spread, (rows, cols // G))
    x = rng.standard_normal((rows, cols)) * np.exp2(np.repeat(blk, G, axis=1))
    zero = np.repeat(rng.random((rows, cols // G)) < zero_frac, G, axis=1)
    return np.where(zero, 0.0, x).astype(np.float32)


def check_compact(x, fmt, dtype, G, S, what):
    if dtype == "bf16":
        x = W.bf16_round(x)
    say(f"[compact] {what} fmt={fmt} dtype={dtype} G={G} S={S} shape={x.shape}")
    codes, ref, offs = cf.curvefp_quantize_compact(to_dev(x, dtype), fmt, G, S)
    scales = cf.curvefp_scales_unpack(ref, offs, x.shape[1] // G, S)
    torch.cuda.synchronize()
    f = oracle.get_format(fmt)
    oc, oref, od = oracle.quantize_compact(x, f, G, S)
    assert np.array_equal(ref.cpu().numpy(), oref), f"{what}: row references differ"
    assert np.array_equal(offs.cpu().numpy(), oracle.pack_offsets(od, S)), f"{what}: packed offsets differ"
    exp_c = layout_codes(oc, fmt)
    got_c = codes.cpu().numpy().reshape(exp_c.shape)
    assert np.array_equal(got_c, exp_c), f"{what}: {np.sum(got_c != exp_c)} code bytes differ"
    assert np.array_equal(scales.cpu().numpy(), oracle.compact_scales(oref, od, S)), f"{what}: unpacked scales"
    return codes, scales, (oc, oracle.compact_scales(oref, od, S))


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("G,S", [(32, 4), (64, 4), (64, 5), (512, 5), (96, 3), (1536, 8), (128, 2)])
def test_quantize_compact(fmt, dtype, G, S):
    rng = np.random.default_rng(G + 10 * S)
    x = spread_rows(rng, 29, 1536, G, 24)
    check_compact(x, fmt, dtype, G, S, "spread")


@pytest.mark.parametrize("fmt", FMTS)
def test_quantize_compact_edges(fmt):
    for kind in W.EDGE_KINDS:
        x = W.edge_tensor(kind, (64, 512))
        check_compact(x, fmt, "f32", 64, 4, kind)
        check_compact(x, fmt, "f32", 128, 5, kind)
    x = W.edge_tensor("nonfinite", (32, 512))
    check_compact(x, fmt, "f32", 64, 4, "nonfinite")
    check_compact(x, fmt, "bf16", 64, 5, "nonfinite")
    # one row, one block; a row of 131072 elements (4096 groups, the limit)
    check_compact(np.linspace(-3, 3, 32, dtype=np.float32).reshape(1, 32), fmt, "f32", 32, 4, "one_block")
    rng = np.random.default_rng(9)
    check_compact(spread_rows(rng, 2, 131072, 512, 20), fmt, "bf16", 512, 5, "long_rows")


@pytest.mark.parametrize("which,S", [("a", 5), ("b", 4)])
def test_inference_operands(which, S):
    """The inference operands in E3C3 with G64 and the paper's scale widths (S = 5 for the
    activation, 4 for the weight)."""
    x = W.get("inference").operand(which)
    check_compact(x, "E3C3", "bf16", 64, S, f"inference_{which}")


@pytest.mark.parametrize("fmt", FMTS)
def test_consumers(fmt):
    """Unpacked S-bit scales feed dequantize and the workspace GEMM like any block scales."""
    M, N, K, G = 160, 200, 1024, 64
    rng = np.random.default_rng(21)
    A = spread_rows(rng, M, K, G, 20, 0.05)
    B = (spread_rows(rng, N, K, G, 20, 0.05) * np.float32(2.0 ** -8)).astype(np.float32)
    ca, sa, (oca, osa) = check_compact(A, fmt, "f32", G, 5, "A")
    cb, sb, (ocb, osb) = check_compact(B, fmt, "f32", G, 4, "B")
    xa = cf.curvefp_dequantize(ca, sa, fmt, M, K, block=G)
    C = cf.curvefp_gemm_ws(ca, sa, cb, sb, M, N, K, fmt, block=G)
    torch.cuda.synchronize()
    f = oracle.get_format(fmt)
    exp = oracle.dequantize(oca, osa, f, G)
    assert np.array_equal(xa.cpu().numpy().view(np.uint32), exp.view(np.uint32))
    V = oracle.gemm_exact(oca, osa, ocb, osb, f, block=G)
    check_gemm(C.cpu().numpy(), V, gemm_tolerance(oca, osa, ocb, osb, fmt, block=G), f"compact gemm {fmt}")
