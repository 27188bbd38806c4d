"""GPU parity for block sizes G other than 32: one scale per G consecutive elements along the
blocked axis (Eq. effective-rate's G; Sec. 3.1 evaluates fixed-size blocks and rowwise sharing,
Sec. 4.2 uses G64 and G512).

* curvefp_quantize, both axes, bit for bit against the oracle: blocks of 64..512 along rows are
  reduced over their lanes in one pass; other G (96, rowwise) and every G down the columns take
  the scale pass first.
* curvefp_dequantize bit for bit against the oracle.
* The GEMM entry points against the exact oracle over blocks of G, and bit for bit against the
  same codes with every scale repeated to blocks of 32: the expanded operand values are the same,
  so the fp32 results must be too.
"""

import numpy as np
import pytest
import torch

import oracle
from paper_2608_10010_amd import curvefp as cf
from paper_2608_10010_amd import workloads as W
from tests.gpu_util import (DEV, FMTS, check_gemm, gemm_tolerance, gemm_tolerance_mixed, layout_codes, say,
                            to_dev)

pytestmark = pytest.mark.gpu

GS = [64, 128, 256, 512, 96]


def source(rng, rows, cols, zero_frac=0.1):
    """Groups of 32 along rows with magnitudes 2^U(-20, 20), some groups all zero."""
    g = np.exp2(rng.uniform(-20, 20, (rows, cols // 32)))
    x = rng.standard_normal((rows, cols)) * np.repeat(g, 32, axis=1)
    zero = rng.random((rows, cols // 32)) < zero_frac
    return np.where(np.repeat(zero, 32, axis=1), 0.0, x).astype(np.float32)


def check_quantize(x, fmt, dtype, axis, G, what):
    if dtype == "bf16":
        x = W.bf16_round(x)
    say(f"[blocks] quantize {what} fmt={fmt} dtype={dtype} axis={axis} G={G} shape={x.shape}")
    codes, scales = cf.curvefp_quantize(to_dev(x, dtype), fmt, block_axis=axis, block=G)
    torch.cuda.synchronize()
    xo = x if axis == 1 else np.ascontiguousarray(x.T)
    oc, os_ = oracle.quantize(xo, oracle.get_format(fmt), G)
    got_s = scales.cpu().numpy()
    assert got_s.shape == os_.shape and np.array_equal(got_s, os_), \
        f"{what}: {np.sum(got_s != os_)} of {os_.size} scales differ"
    exp_c = layout_codes(oc, fmt)
    got_c = codes.cpu().numpy().reshape(exp_c.shape)
    assert np.array_equal(got_c, exp_c), f"{what}: {np.sum(got_c != exp_c)} code bytes differ"
    return codes, scales


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("G", GS + ["row"])
def test_quantize_rows(fmt, dtype, G):
    rng = np.random.default_rng(100 + (G if G != "row" else 1))
    rows, cols = 37, 1536
    G = cols if G == "row" else G
    check_quantize(source(rng, rows, cols), fmt, dtype, 1, G, "rows")


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("G", GS + ["col"])
@pytest.mark.parametrize("cols", [45, 72])
def test_quantize_cols(fmt, G, cols):
    # 45 columns: one thread per 32-row block; 72 columns (rows % 128 == 0, cols % 8 == 0): the
    # LDS-tiled transpose with a last tile of 8 columns
    rng = np.random.default_rng(200 + cols + (G if G != "col" else 2))
    rows = 1536
    G = rows if G == "col" else G
    x = np.ascontiguousarray(source(rng, cols, rows).T)     # groups of 32 down the columns
    check_quantize(x, fmt, "bf16" if cols == 72 else "f32", 0, G, "cols")


@pytest.mark.parametrize("fmt", FMTS)
def test_quantize_edges(fmt):
    for kind in W.EDGE_KINDS:
        x = W.edge_tensor(kind, (64, 512))
        check_quantize(x, fmt, "f32", 1, 128, kind)
        check_quantize(x, fmt, "f32", 1, 512, kind)
        check_quantize(np.ascontiguousarray(x.T), fmt, "f32", 0, 64, kind + "_T")
    x = W.edge_tensor("nonfinite", (32, 512))
    for G in (64, 256, 512):
        check_quantize(x, fmt, "f32", 1, G, "nonfinite")
        check_quantize(x, fmt, "bf16", 1, G, "nonfinite")
    check_quantize(np.ascontiguousarray(x[:, :256].T), fmt, "f32", 0, 128, "nonfinite_T")


@pytest.mark.parametrize("G", [512, 4096])
def test_quantize_inference_activation_blocks(G):
    """The inference activation (2048 x 4096 bf16, outlier channels) with G512 and rowwise
    scales, in E3C3 (the paper's G sweep format)."""
    a = W.get("inference").operand("a")
    check_quantize(a, "E3C3", "bf16", 1, G, "inference_act")


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("G", [64, 512, 96, 1536])
def test_dequantize(fmt, G):
    rng = np.random.default_rng(300 + G)
    x = source(rng, 21, 1536)
    f = oracle.get_format(fmt)
    oc, os_ = oracle.quantize(x, f, G)
    say(f"[blocks] dequantize fmt={fmt} G={G}")
    codes = torch.from_numpy(np.ascontiguousarray(layout_codes(oc, fmt))).to(DEV)
    scales = torch.from_numpy(os_).to(DEV)
    out = cf.curvefp_dequantize(codes, scales, fmt, 21, 1536, block=G)
    torch.cuda.synchronize()
    exp = oracle.dequantize(oc, os_, f, G)
    got = out.cpu().numpy()
    assert np.array_equal(got.view(np.uint32), exp.view(np.uint32))


def same_bits(x, y, what):
    assert x.shape == y.shape
    bad = x.view(np.uint32) != y.view(np.uint32)
    assert not bad.any(), f"{what}: {bad.sum()} elements differ"


def repeat32(scales: torch.Tensor, G: int) -> torch.Tensor:
    return torch.repeat_interleave(scales, G // 32, dim=1).contiguous()


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("G,shape", [(64, (200, 136, 1536)), (512, (200, 136, 1536)), (96, (130, 260, 1536)),
                                     (1536, (64, 300, 1536)), (2048, (96, 80, 2048)), (512, (256, 256, 4096))])
def test_gemm(fmt, G, shape):
    M, N, K = shape
    rng = np.random.default_rng(M + N + K + G)
    A = source(rng, M, K, 0.05)
    B = (source(rng, N, K, 0.05) * np.float32(2.0 ** -12)).astype(np.float32)
    say(f"[blocks] gemm fmt={fmt} G={G} M={M} N={N} K={K}")
    qa = cf.curvefp_quantize(to_dev(A, "f32"), fmt, block=G)
    qb = cf.curvefp_quantize(to_dev(B, "f32"), fmt, block=G)
    Cw = cf.curvefp_gemm_ws(qa[0], qa[1], qb[0], qb[1], M, N, K, fmt, block=G)
    Cf = cf.curvefp_gemm(qa[0], qa[1], qb[0], qb[1], M, N, K, fmt, block=G)
    C32 = cf.curvefp_gemm_ws(qa[0], repeat32(qa[1], G), qb[0], repeat32(qb[1], G), M, N, K, fmt)
    torch.cuda.synchronize()
    Cw, Cf, C32 = Cw.cpu().numpy(), Cf.cpu().numpy(), C32.cpu().numpy()
    same_bits(Cw, C32, f"ws G={G} vs G=32 repeated")
    same_bits(Cf, Cw, f"fused G={G} vs ws")
    f = oracle.get_format(fmt)
    ca, sa = oracle.quantize(A, f, G)
    cb, sb = oracle.quantize(B, f, G)
    V = oracle.gemm_exact(ca, sa, cb, sb, f, block=G)
    check_gemm(Cw, V, gemm_tolerance(ca, sa, cb, sb, fmt, block=G), f"ws {fmt} G={G} {shape}")


@pytest.mark.parametrize("fmt,ofmt", [("E3C3", "E3C3"), ("E4C3", "E5C2"), ("E4C3_r3/4", "E4C3")])
@pytest.mark.parametrize("G", [64, 512])
def test_gemm_requant(fmt, ofmt, G):
    M, N, K = 200, 320, 2048
    rng = np.random.default_rng(400 + G)
    A = source(rng, M, K, 0.05)
    B = (source(rng, N, K, 0.05) * np.float32(2.0 ** -12)).astype(np.float32)
    say(f"[blocks] requant fmt={fmt} out={ofmt} G={G}")
    qa = cf.curvefp_quantize(to_dev(A, "f32"), fmt, block=G)
    qb = cf.curvefp_quantize(to_dev(B, "f32"), fmt, block=G)
    oc, os_ = cf.curvefp_gemm_requant(qa[0], qa[1], qb[0], qb[1], M, N, K, fmt, ofmt, block=G)
    C = cf.curvefp_gemm_ws(qa[0], qa[1], qb[0], qb[1], M, N, K, fmt, block=G)
    rc, rs = cf.curvefp_quantize(C, ofmt)
    torch.cuda.synchronize()
    assert np.array_equal(os_.cpu().numpy(), rs.cpu().numpy())
    assert np.array_equal(oc.cpu().numpy(), rc.cpu().numpy())


@pytest.mark.parametrize("ta,tb", [(0, 1), (1, 1), (0, 0)])
@pytest.mark.parametrize("G", [64, 256])
def test_gemm_mixed(ta, tb, G):
    """The backward recipe (E5C2 x reused E4C3 codes) with blocks of G; a reused operand's
    blocks run along its GEMM rows."""
    fa, fb = "E5C2", "E4C3"
    M, N, K = 256, 512, 512
    rng = np.random.default_rng(500 + G + 2 * ta + tb)
    # a reused operand's source is [K][R] quantized along R; one quantized along K is [R][K]
    A = source(rng, K, M) if ta else source(rng, M, K)
    B = (source(rng, K, N) if tb else source(rng, N, K)) * np.float32(2.0 ** -10)
    say(f"[blocks] mixed ta={ta} tb={tb} G={G}")
    qa = cf.curvefp_quantize(to_dev(A, "f32"), fa, block=G)
    qb = cf.curvefp_quantize(to_dev(B.astype(np.float32), "f32"), fb, block=G)
    C = cf.curvefp_gemm_mixed(qa[0], qa[1], fa, ta, qb[0], qb[1], fb, tb, M, N, K, block=G)
    C32 = cf.curvefp_gemm_mixed(qa[0], repeat32(qa[1], G), fa, ta, qb[0], repeat32(qb[1], G), fb, tb, M, N, K)
    torch.cuda.synchronize()
    C, C32 = C.cpu().numpy(), C32.cpu().numpy()
    same_bits(C, C32, f"mixed G={G} vs G=32 repeated")

    def operand(X, fmt, trans):
        c, s = oracle.quantize(X, oracle.get_format(fmt), G)
        if not trans:
            return c, oracle.expand_scales(s, G, axis=1)
        return np.ascontiguousarray(c.T), oracle.expand_scales(s, G, axis=0)

    ca, sa = operand(A, fa, ta)
    cb, sb = operand(B.astype(np.float32), fb, tb)
    V = oracle.gemm_exact_mixed(ca, sa, oracle.get_format(fa), cb, sb, oracle.get_format(fb))
    check_gemm(C, V, gemm_tolerance_mixed(ca, sa, fa, cb, sb, fb), f"mixed ta={ta} tb={tb} G={G}")


@pytest.mark.parametrize("G", [512, 4096])
def test_inference_full_size(G):
    """The inference workload at its full size (2048 x 4096 x 4096 E3C3, bf16 sources) with G512
    and rowwise scales, in the launch configuration bench.py times: the workspace GEMM equals the
    G = 32 call on the same codes with repeated scales bit for bit, and 16 sampled rows equal the
    exact oracle on the oracle's own quantization within the bound."""
    w = W.get("inference")
    A, B = w.operand("a"), w.operand("b")
    say(f"[blocks] inference full size G={G}")
    qa = cf.curvefp_quantize(to_dev(A, "bf16"), w.fmt, block=G)
    qb = cf.curvefp_quantize(to_dev(B, "bf16"), w.fmt, block=G)
    C = cf.curvefp_gemm_ws(qa[0], qa[1], qb[0], qb[1], w.M, w.N, w.K, w.fmt, block=G)
    C32 = cf.curvefp_gemm_ws(qa[0], repeat32(qa[1], G), qb[0], repeat32(qb[1], G), w.M, w.N, w.K, w.fmt)
    torch.cuda.synchronize()
    C = C.cpu().numpy()
    same_bits(C, C32.cpu().numpy(), f"inference G={G} vs G=32 repeated")
    f = oracle.get_format(w.fmt)
    rows = np.random.default_rng(G).choice(w.M, 16, replace=False)
    ca, sa = oracle.quantize(np.ascontiguousarray(A[rows]), f, G)
    cb, sb = oracle.quantize(B, f, G)
    V = oracle.gemm_exact(ca, sa, cb, sb, f, block=G)
    check_gemm(C[rows], V, gemm_tolerance(ca, sa, cb, sb, w.fmt, block=G), f"inference G={G} sampled rows")
