"""GPU parity of curvefp_quantize_prepare (quantize, prepare and reconstruct in one launch): codes and
scales bit-exact against the oracle's quantizer and the reconstruction against the oracle's
dequantizer; codes, scales, prepared bytes and reconstruction identical to curvefp_quantize,
curvefp_prepare and curvefp_dequantize on the same source; products of fused-prepared operands
identical to curvefp_gemm_ws and within the GEMM bound of the exact phase-binned oracle.  Shapes span
every row length class (a wave or a workgroup per row, with 2, 4 or 8 chunks per lane staged in LDS;
longer rows through the separate kernels), padding rows up to the next tile of 256, blocks of
32 .. 512, row strides, the edge tensors and non-finite blocks."""

import numpy as np
import pytest
import torch

import oracle
from paper_2608_10010_amd import curvefp as cf
from paper_2608_10010_amd import workloads as W
from tests.gpu_util import DEV, FMTS, check_gemm, gemm_tolerance, layout_codes, say, to_dev
from tests.test_gpu_gemm_ws import same_bits

pytestmark = pytest.mark.gpu


def same_bytes(x: torch.Tensor, y: torch.Tensor, what: str):
    a, b = x.contiguous().view(torch.uint8), y.contiguous().view(torch.uint8)
    assert a.shape == b.shape, what
    bad = int((a != b).sum())
    assert bad == 0, f"{what}: {bad} bytes differ"


def fused_vs_separate(t: torch.Tensor, fmt: str, block: int, what: str, ld_dst_pad: int = 0):
    """The fused call against the three separate calls on the same source, byte for byte."""
    rows, k = t.shape
    say(f"[quantize_prepare] {what} fmt={fmt} dtype={t.dtype} rows={rows} k={k} G={block}")
    dst = None
    if ld_dst_pad:
        dst = torch.full((rows, k + ld_dst_pad), 3.0, dtype=torch.float32, device=DEV)[:, :k]
    codes, scales, prep, d = cf.curvefp_quantize_prepare(t, fmt, block=block, dst=dst, dequantize=True)
    c0, s0, p0 = cf.curvefp_quantize_prepare(t, fmt, block=block)          # without the reconstruction
    c2, s2 = cf.curvefp_quantize(t, fmt, block=block)
    p2 = cf.curvefp_prepare(c2, s2, rows, k, fmt, block=block)
    d2 = cf.curvefp_dequantize(c2, s2, fmt, rows, k, block=block)
    torch.cuda.synchronize()
    for x, y, n in ((codes, c2, "codes"), (scales, s2, "scales"), (prep, p2, "prepared"), (d, d2, "dequantized"),
                    (c0, c2, "codes (no reconstruction)"), (s0, s2, "scales (no reconstruction)"),
                    (p0, p2, "prepared (no reconstruction)")):
        same_bytes(x, y, f"{what} {fmt}: {n}")
    if ld_dst_pad:
        pad = dst.as_strided((rows, ld_dst_pad), (dst.stride(0), 1), dst.storage_offset() + k)
        assert bool((pad == 3.0).all()), f"{what}: wrote past the rows of dst"
    return codes, scales, prep, d


def oracle_check(x: np.ndarray, fmt: str, block: int, codes, scales, d, what: str):
    f = oracle.get_format(fmt)
    oc, os_ = oracle.quantize(x, f, block)
    assert np.array_equal(scales.cpu().numpy(), os_), f"{what}: scales differ from the oracle"
    got = codes.cpu().numpy()
    exp = layout_codes(oc, fmt)
    assert np.array_equal(got.reshape(exp.shape), exp), f"{what}: codes differ from the oracle"
    od = oracle.dequantize(oc, os_, f, block)
    assert np.array_equal(d.cpu().numpy().view(np.uint32), od.view(np.uint32)), \
        f"{what}: reconstruction differs from the oracle"


def source(x: np.ndarray, dtype: str) -> torch.Tensor:
    return to_dev(x, dtype)


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("rows,k,block", [(1, 32, 32), (37, 352, 32), (300, 1024, 64), (70, 2048, 128),
                                          (257, 4096, 512), (9, 4096, 256)])
def test_random(fmt, dtype, rows, k, block):
    rng = np.random.default_rng(rows * 131 + k + block)
    x = (rng.standard_normal((rows, k)) * np.exp2(rng.uniform(-30, 30, (rows, 1)))).astype(np.float32)
    if dtype == "bf16":
        x = W.bf16_round(x)
    codes, scales, _, d = fused_vs_separate(source(x, dtype), fmt, block, "random")
    oracle_check(x, fmt, block, codes, scales, d, f"random {rows}x{k} G{block}")


@pytest.mark.parametrize("fmt", ["E4C3", "E3C3", "E5C2"])
@pytest.mark.parametrize("dtype,k", [("bf16", 32768), ("bf16", 16384), ("bf16", 14336), ("bf16", 8224), ("bf16", 8192),
                                     ("bf16", 4160), ("f32", 8192), ("f32", 4128), ("f32", 4096), ("f32", 2080)])
def test_long_rows(fmt, dtype, k):
    """Rows staged per workgroup (whole and partial segments), and rows too long for that (the three
    kernels in turn)."""
    rows = 40 if k <= 16384 else 8
    rng = np.random.default_rng(k)
    x = (rng.standard_normal((rows, k)) * np.exp2(rng.uniform(-8, 8, (rows, k // 32)).repeat(32, axis=1))).astype(
        np.float32)
    if dtype == "bf16":
        x = W.bf16_round(x)
    for block in (32, 256) if k % 256 == 0 else (32,):
        codes, scales, _, d = fused_vs_separate(source(x, dtype), fmt, block, f"long k={k}")
        oracle_check(x, fmt, block, codes, scales, d, f"long k={k} G{block}")


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("kind", W.EDGE_KINDS)
def test_edges(fmt, dtype, kind):
    x = W.edge_tensor(kind, (64, 256))
    if dtype == "bf16":
        x = W.bf16_round(x)
    codes, scales, _, d = fused_vs_separate(source(x, dtype), fmt, 32, kind)
    oracle_check(x, fmt, 32, codes, scales, d, kind)


@pytest.mark.parametrize("fmt", FMTS)
def test_nonfinite_poison(fmt):
    x = W.edge_tensor("nonfinite", (32, 512))
    for dtype in ("f32", "bf16"):
        xs = W.bf16_round(x) if dtype == "bf16" else x
        codes, scales, prep, d = fused_vs_separate(source(xs, dtype), fmt, 32, f"nonfinite {dtype}")
        oracle_check(xs, fmt, 32, codes, scales, d, f"nonfinite {dtype}")


@pytest.mark.parametrize("fmt", ["E4C3", "E3C3"])
def test_row_strides(fmt):
    rng = np.random.default_rng(3)
    x = rng.standard_normal((100, 512)).astype(np.float32)
    full = to_dev(np.concatenate([x, np.full((100, 64), 9.0, np.float32)], axis=1), "bf16")
    t = full[:, :512]
    codes, scales, _, d = fused_vs_separate(t, fmt, 32, "strided", ld_dst_pad=40)
    oracle_check(W.bf16_round(x), fmt, 32, codes, scales, d, "strided")


@pytest.mark.parametrize("fmt", ["E4C3", "E5C2", "E3C3", "E4C3_r3/4"])
@pytest.mark.parametrize("shape", [(300, 520, 640), (64, 300, 1024), (1, 1, 32)])
def test_gemm_on_fused_operands(fmt, shape):
    """Both operands quantized and prepared in one launch each: the prepared GEMM equals the workspace
    GEMM on the same codes bit for bit, and the exact oracle within the GEMM bound."""
    M, N, K = shape
    rng = np.random.default_rng(M + N + K)
    A = W.bf16_round((rng.standard_normal((M, K)) * np.exp2(rng.uniform(-6, 6, (M, 1)))).astype(np.float32))
    B = W.bf16_round((rng.standard_normal((N, K)) * 0.02).astype(np.float32))
    say(f"[quantize_prepare] gemm fmt={fmt} M={M} N={N} K={K}")
    ca, sa, pa = cf.curvefp_quantize_prepare(to_dev(A, "bf16"), fmt)
    cb, sb, pb = cf.curvefp_quantize_prepare(to_dev(B, "bf16"), fmt)
    C = cf.curvefp_gemm_prepared(pa, fmt, pb, fmt, M, N, K)
    Cw = cf.curvefp_gemm_ws(ca, sa, cb, sb, M, N, K, fmt)
    torch.cuda.synchronize()
    C, Cw = C.cpu().numpy(), Cw.cpu().numpy()
    same_bits(C, Cw, f"fused-prepared {fmt} {shape}")
    f = oracle.get_format(fmt)
    oca, osa = oracle.quantize(A, f)
    ocb, osb = oracle.quantize(B, f)
    V = oracle.gemm_exact(oca, osa, ocb, osb, f)
    check_gemm(C, V, gemm_tolerance(oca, osa, ocb, osb, fmt), f"fused-prepared {fmt} {shape}")


@pytest.mark.parametrize("name", ["sweep_gateup_E4C3", "sweep_down_E3C3"])
def test_workload_full_size(name):
    """The benchmark's operands at full size: the fused call equals the separate ones byte for byte,
    sampled rows match the oracle, and the product of fused-prepared operands equals the workspace
    GEMM bit for bit."""
    w = W.get(name)
    ta = torch.from_numpy(w.operand("a")).to(torch.bfloat16).to(DEV)
    tb = torch.from_numpy(w.operand("b")).to(torch.bfloat16).to(DEV)
    ca, sa, pa, da = fused_vs_separate(ta, w.fmt, 32, name + " act")
    cb, sb, pb = cf.curvefp_quantize_prepare(tb, w.fmt)
    rows = np.array([0, 1, 255, 256, w.M // 2, w.M - 1])
    xa = ta[torch.from_numpy(rows).to(DEV)].float().cpu().numpy()
    oracle_check(xa, w.fmt, 32, ca[torch.from_numpy(rows).to(DEV)], sa[torch.from_numpy(rows).to(DEV)],
                 da[torch.from_numpy(rows).to(DEV)], name + " sampled rows")
    del ta, tb, da
    C = cf.curvefp_gemm_prepared(pa, w.fmt, pb, w.fmt, w.M, w.N, w.K)
    Cw = cf.curvefp_gemm_ws(ca, sa, cb, sb, w.M, w.N, w.K, w.fmt)
    torch.cuda.synchronize()
    assert torch.equal(C.view(torch.int32), Cw.view(torch.int32)), f"{name}: fused-prepared GEMM differs"


@pytest.mark.parametrize("fmt", ["E4C3", "E5C2", "E3C3", "E4C3_r8/9"])
@pytest.mark.parametrize("dtype,ra,rb,k,block", [("bf16", 300, 520, 640, 32), ("bf16", 1, 257, 4096, 64),
                                                  ("f32", 129, 64, 2048, 128), ("bf16", 40, 24, 8192, 32),
                                                  ("bf16", 16, 8, 32768, 32)])
def test_pair(fmt, dtype, ra, rb, k, block):
    """Both operands in one launch (a wave or a workgroup per row, or the separate kernels for the
    longest rows): the outputs of two single calls, byte for byte, and the GEMM on them that of the
    workspace GEMM."""
    rng = np.random.default_rng(ra * 7 + rb + k)
    A = (rng.standard_normal((ra, k)) * np.exp2(rng.uniform(-20, 20, (ra, 1)))).astype(np.float32)
    B = (rng.standard_normal((rb, k)) * 0.02).astype(np.float32)
    if dtype == "bf16":
        A, B = W.bf16_round(A), W.bf16_round(B)
    ta, tb = source(A, dtype), source(B, dtype)
    say(f"[quantize_prepare] pair fmt={fmt} dtype={dtype} rows={ra}+{rb} k={k} G={block}")
    pa, pb = cf.curvefp_quantize_prepare_pair(ta, tb, fmt, block=block, dequantize_a=True)
    sa_ = cf.curvefp_quantize_prepare(ta, fmt, block=block, dequantize=True)
    sb_ = cf.curvefp_quantize_prepare(tb, fmt, block=block)
    torch.cuda.synchronize()
    assert len(pa) == 4 and len(pb) == 3
    for x, y, n in zip(pa + pb, sa_ + sb_, ("codes A", "scales A", "prepared A", "dst A", "codes B", "scales B",
                                            "prepared B")):
        same_bytes(x, y, f"pair {fmt} {ra}+{rb}x{k}: {n}")
    oracle_check(A, fmt, block, pa[0], pa[1], pa[3], f"pair {fmt} A")
    if k <= 8192:
        C = cf.curvefp_gemm_prepared(pa[2], fmt, pb[2], fmt, ra, rb, k)
        Cw = cf.curvefp_gemm_ws(pa[0], pa[1], pb[0], pb[1], ra, rb, k, fmt, block=block)
        torch.cuda.synchronize()
        same_bits(C.cpu().numpy(), Cw.cpu().numpy(), f"pair {fmt} gemm")


@pytest.mark.parametrize("dtype,k", [("bf16", 1024), ("f32", 4096), ("bf16", 8192)])
def test_pair_both_reconstructed(dtype, k):
    """Both operands with their reconstruction (the second operand's dst included), against single
    calls byte for byte and against the oracle."""
    ra, rb = 70, 33
    rng = np.random.default_rng(k + 3)
    A = (rng.standard_normal((ra, k)) * np.exp2(rng.uniform(-30, 30, (ra, 1)))).astype(np.float32)
    B = (rng.standard_normal((rb, k)) * np.exp2(rng.uniform(-30, 30, (rb, 1)))).astype(np.float32)
    if dtype == "bf16":
        A, B = W.bf16_round(A), W.bf16_round(B)
    ta, tb = source(A, dtype), source(B, dtype)
    say(f"[quantize_prepare] pair, both reconstructed, dtype={dtype} rows={ra}+{rb} k={k}")
    pa, pb = cf.curvefp_quantize_prepare_pair(ta, tb, "E3C3", dequantize_a=True, dequantize_b=True)
    sa_ = cf.curvefp_quantize_prepare(ta, "E3C3", dequantize=True)
    sb_ = cf.curvefp_quantize_prepare(tb, "E3C3", dequantize=True)
    torch.cuda.synchronize()
    assert len(pa) == 4 and len(pb) == 4
    for x, y, n in zip(pa + pb, sa_ + sb_, ("codes A", "scales A", "prepared A", "dst A", "codes B", "scales B",
                                            "prepared B", "dst B")):
        same_bytes(x, y, f"pair both reconstructed {dtype} k={k}: {n}")
    oracle_check(A, "E3C3", 32, pa[0], pa[1], pa[3], "pair both reconstructed A")
    oracle_check(B, "E3C3", 32, pb[0], pb[1], pb[3], "pair both reconstructed B")


@pytest.mark.parametrize("k", [512, 4096])
def test_pair_row_strides(k):
    """Both operands read from row-strided views and reconstructed into row-strided outputs: the
    padding columns of the sources are never read and those of the outputs never written."""
    ra, rb = 45, 130
    rng = np.random.default_rng(k)
    A = W.bf16_round(rng.standard_normal((ra, k)).astype(np.float32))
    B = W.bf16_round((rng.standard_normal((rb, k)) * 0.02).astype(np.float32))
    fa = to_dev(np.concatenate([A, np.full((ra, 64), 7.0e30, np.float32)], axis=1), "bf16")
    fb = to_dev(np.concatenate([B, np.full((rb, 32), -3.0e30, np.float32)], axis=1), "bf16")
    ta, tb = fa[:, :k], fb[:, :k]
    da = torch.full((ra, k + 16), 5.0, dtype=torch.float32, device=DEV)
    db = torch.full((rb, k + 8), 6.0, dtype=torch.float32, device=DEV)
    say(f"[quantize_prepare] pair on row-strided views k={k}")
    pa, pb = cf.curvefp_quantize_prepare_pair(ta, tb, "E4C3", out_a=(None, None, None, da[:, :k]),
                                              out_b=(None, None, None, db[:, :k]))
    sa_ = cf.curvefp_quantize_prepare(ta.contiguous(), "E4C3", dequantize=True)
    sb_ = cf.curvefp_quantize_prepare(tb.contiguous(), "E4C3", dequantize=True)
    torch.cuda.synchronize()
    for x, y, n in zip(pa + pb, sa_ + sb_, ("codes A", "scales A", "prepared A", "dst A", "codes B", "scales B",
                                            "prepared B", "dst B")):
        same_bytes(x, y, f"strided pair k={k}: {n}")
    assert bool((da[:, k:] == 5.0).all()) and bool((db[:, k:] == 6.0).all()), "padding columns written"
    oracle_check(A, "E4C3", 32, pa[0], pa[1], pa[3], "strided pair A")
    oracle_check(B, "E4C3", 32, pb[0], pb[1], pb[3], "strided pair B")


def test_pair_benchmark_operands():
    """The benchmark's step: both gate/up operands in one launch equal two single calls."""
    w = W.get("sweep_gateup_E4C3")
    ta = torch.from_numpy(w.operand("a")).to(torch.bfloat16).to(DEV)
    tb = torch.from_numpy(w.operand("b")).to(torch.bfloat16).to(DEV)
    say("[quantize_prepare] pair on the gate/up operands")
    pa, pb = cf.curvefp_quantize_prepare_pair(ta, tb, w.fmt, dequantize_a=True)
    sa_ = cf.curvefp_quantize_prepare(ta, w.fmt, dequantize=True)
    sb_ = cf.curvefp_quantize_prepare(tb, w.fmt)
    torch.cuda.synchronize()
    for x, y, n in zip(pa + pb, sa_ + sb_, ("codes A", "scales A", "prepared A", "dst A", "codes B", "scales B",
                                            "prepared B")):
        same_bytes(x, y, f"gate/up pair: {n}")


def test_pair_too_large_together():
    """Operands of 16384-element rows too large to share a launch (over 2^26 elements together):
    each is taken on its own -- the larger by the separate kernels, the smaller by the fused one --
    with the outputs of two single calls, byte for byte."""
    ra, rb, k = 5000, 1000, 16384
    g = torch.Generator(device=DEV)
    g.manual_seed(9)
    ta = (torch.randn((ra, k), generator=g, device=DEV) * 3.0).to(torch.bfloat16)
    tb = (torch.randn((rb, k), generator=g, device=DEV) * 0.02).to(torch.bfloat16)
    say(f"[quantize_prepare] pair too large together rows={ra}+{rb} k={k}")
    pa, pb = cf.curvefp_quantize_prepare_pair(ta, tb, "E4C3", dequantize_a=True)
    sa_ = cf.curvefp_quantize_prepare(ta, "E4C3", dequantize=True)
    sb_ = cf.curvefp_quantize_prepare(tb, "E4C3")
    torch.cuda.synchronize()
    for x, y, n in zip(pa + pb, sa_ + sb_, ("codes A", "scales A", "prepared A", "dst A", "codes B", "scales B",
                                            "prepared B")):
        same_bytes(x, y, f"large pair: {n}")
    rows = torch.tensor([0, 1, 2500, ra - 1], device=DEV)
    xa = ta[rows].float().cpu().numpy()
    oracle_check(xa, "E4C3", 32, pa[0][rows], pa[1][rows], pa[3][rows], "large pair A sampled rows")
    rows_b = torch.tensor([0, rb - 1], device=DEV)
    xb = tb[rows_b].float().cpu().numpy()
    f = oracle.get_format("E4C3")
    oc, os_ = oracle.quantize(xb, f)
    assert np.array_equal(pb[1][rows_b].cpu().numpy(), os_) and np.array_equal(pb[0][rows_b].cpu().numpy(), oc)
