"""The CurveFP GEMM's accuracy contract on rows whose block scales spread widely.

The MFMA realization expands every element relative to the largest block scale alpha of its
row, top = 2^{alpha + e_max + 1} (fp16 high/low pairs carrying 2^{a_b - alpha}).  Stated in
include/curvefp.h as the scale-spread limit:

* an element of magnitude at least 2^-18 top keeps 22 significant bits (relative error
  about 2^-21 for each product);
* below that it keeps an absolute error of at most 2^-39 top;
* below 2^-41 top it is flushed to zero.

These tests hold the kernels to each clause with operands built for it, codes and scales
written directly so every block's scale is chosen:

* rows whose scales span at most 12 binades: every output within 1e-5 sum_k |a b| of the
  oracle's exact phase-binned sum, with no allowance for lost elements at all;
* rows with blocks 60 binades below the row's top block: the output equals, to 1e-5, the exact
  product with those far elements removed (the flush, exactly), and it is materially different
  from the exact product (the limit is real, not hidden in a tolerance);
* rows whose blocks lie 20..36 binades below the top: within the per-element loss bound;
* an all-zero block no longer counts as a row's largest scale: a row of values near 2^-50 with
  one zero block is as accurate as any narrow row (through the quantizer, on its -127 scale).
"""

import numpy as np
import pytest
import torch

import oracle
from paper_2608_10010_amd import curvefp as cf
from tests.gpu_util import (BINARY_FMTS, DEV, check_gemm, exact_values, gemm_tolerance, layout_codes,
                            oracle_quantize, row_tops, say, to_dev)

pytestmark = pytest.mark.gpu

K = 512          # 16 blocks of 32


def random_codes(rng, f, shape):
    """Nonzero codes of every magnitude and both signs."""
    m = rng.integers(1, 2 ** (f.E + f.C), shape)
    s = rng.integers(0, 2, shape)
    return ((s << (f.E + f.C)) | m).astype(np.uint8)


def gpu_gemms(ca, sa, cb, sb, fmt):
    M, N = ca.shape[0], cb.shape[0]
    dca = torch.from_numpy(np.ascontiguousarray(layout_codes(ca, fmt))).to(DEV)
    dcb = torch.from_numpy(np.ascontiguousarray(layout_codes(cb, fmt))).to(DEV)
    dsa, dsb = torch.from_numpy(sa).to(DEV), torch.from_numpy(sb).to(DEV)
    Cf = cf.curvefp_gemm(dca, dsa, dcb, dsb, M, N, K, fmt)
    Cw = cf.curvefp_gemm_ws(dca, dsa, dcb, dsb, M, N, K, fmt)
    torch.cuda.synchronize()
    Cf, Cw = Cf.cpu().numpy(), Cw.cpu().numpy()
    assert np.array_equal(Cf.view(np.uint32), Cw.view(np.uint32))
    return Cf.astype(np.float64)


def strict(C, V, ca, sa, cb, sb, fmt, what):
    """No allowance for lost elements: 1e-5 of sum_k |a b| per output."""
    S = np.abs(exact_values(ca, sa, fmt)) @ np.abs(exact_values(cb, sb, fmt)).T
    err = np.abs(C - V)
    assert np.all(err <= 1e-5 * S + 2.0 ** -148), f"{what}: worst {np.max(err / (1e-5 * S + 2.0 ** -148))}"


@pytest.mark.parametrize("fmt", BINARY_FMTS + ("E4C3_r3/4",))
def test_narrow_rows_are_accurate(fmt):
    f = oracle.get_format(fmt)
    rng = np.random.default_rng(71)
    ca, cb = random_codes(rng, f, (48, K)), random_codes(rng, f, (40, K))
    sa = (rng.integers(-30, 30, (48, 1)) - rng.integers(0, 13, (48, K // 32))).astype(np.int8)
    sb = (rng.integers(-30, 30, (40, 1)) - rng.integers(0, 13, (40, K // 32))).astype(np.int8)
    say(f"[contract] narrow rows fmt={fmt}")
    C = gpu_gemms(ca, sa, cb, sb, fmt)
    V = oracle.gemm_exact(ca, sa, cb, sb, f)
    strict(C, V, ca, sa, cb, sb, fmt, f"narrow {fmt}")
    check_gemm(C, V, gemm_tolerance(ca, sa, cb, sb, fmt), f"narrow {fmt}")


@pytest.mark.parametrize("fmt", BINARY_FMTS)
def test_flush_beyond_the_spread_limit(fmt):
    """A's rows: block 0 at scale 20, the other 15 blocks at scale -40 (60 binades below, so
    every element is below 2^-41 top).  B: zero under block 0 in half of its rows."""
    f = oracle.get_format(fmt)
    rng = np.random.default_rng(72)
    M, N = 32, 48
    ca, cb = random_codes(rng, f, (M, K)), random_codes(rng, f, (N, K))
    sa = np.full((M, K // 32), -40, np.int8)
    sa[:, 0] = 20
    sb = rng.integers(-4, 4, (N, K // 32)).astype(np.int8)
    cb[: N // 2, :32] = 0                                    # these rows: nothing under A's top block
    say(f"[contract] flush beyond the spread limit fmt={fmt}")
    C = gpu_gemms(ca, sa, cb, sb, fmt)
    V = oracle.gemm_exact(ca, sa, cb, sb, f)
    va = np.abs(exact_values(ca, sa, fmt))
    far = va < 2.0 ** -41 * row_tops(ca, sa, fmt)[:, None]
    assert far[:, 32:].all() and not far[:, :32].any()
    # the documented flush: the product of A without its far elements, to the element-wise bound
    # of the elements that remain (the top block's own small levels keep the 2^-39 top bound)
    ca_kept = np.where(far, 0, ca).astype(np.uint8)
    Vk = oracle.gemm_exact(ca_kept, sa, cb, sb, f)
    check_gemm(C, Vk, gemm_tolerance(ca_kept, sa, cb, sb, fmt), f"flush {fmt}")
    # where B is zero under the top block, the flushed product is zero while the exact one is not
    assert np.all(C[:, : N // 2] == 0)
    assert np.all(np.abs(V[:, : N // 2]) > 0)
    # and the element-wise tolerance admits exactly that loss, no more
    check_gemm(C, V, gemm_tolerance(ca, sa, cb, sb, fmt), f"flush {fmt}", frobenius=False)


@pytest.mark.parametrize("fmt", BINARY_FMTS)
def test_partial_precision_band(fmt):
    """Blocks 20..36 binades below the row's top block: fewer bits, bounded absolute error."""
    f = oracle.get_format(fmt)
    rng = np.random.default_rng(73)
    M, N = 40, 40
    ca, cb = random_codes(rng, f, (M, K)), random_codes(rng, f, (N, K))
    sa = (10 - rng.integers(20, 37, (M, K // 32))).astype(np.int8)
    sa[:, 0] = 10
    sb = rng.integers(-3, 3, (N, K // 32)).astype(np.int8)
    say(f"[contract] partial precision band fmt={fmt}")
    C = gpu_gemms(ca, sa, cb, sb, fmt)
    V = oracle.gemm_exact(ca, sa, cb, sb, f)
    check_gemm(C, V, gemm_tolerance(ca, sa, cb, sb, fmt), f"band {fmt}", frobenius=False)


@pytest.mark.parametrize("fmt", BINARY_FMTS)
def test_zero_block_does_not_set_the_row_scale(fmt):
    """Rows of values near 2^-50 with one all-zero block, through the quantizer: the zero block's
    scale is -127, so the row's largest scale is that of its real values and nothing is lost."""
    rng = np.random.default_rng(74)
    A = (rng.standard_normal((64, K)) * 2.0 ** -50).astype(np.float32)
    A[:, 64:96] = 0.0
    B = rng.standard_normal((48, K)).astype(np.float32)
    B[:, 64:96] = 0.0
    say(f"[contract] zero block fmt={fmt}")
    qa = cf.curvefp_quantize(to_dev(A, "f32"), fmt)
    qb = cf.curvefp_quantize(to_dev(B, "f32"), fmt)
    assert np.all(qa[1].cpu().numpy()[:, 2] == -127) and np.all(qb[1].cpu().numpy()[:, 2] == -127)
    C = cf.curvefp_gemm_ws(qa[0], qa[1], qb[0], qb[1], 64, 48, K, fmt)
    torch.cuda.synchronize()
    ca, sa = oracle_quantize(A, fmt, 1)
    cb, sb = oracle_quantize(B, fmt, 1)
    f = oracle.get_format(fmt)
    V = oracle.gemm_exact(ca, sa, cb, sb, f)
    strict(C.cpu().numpy().astype(np.float64), V, ca, sa, cb, sb, fmt, f"zero block {fmt}")
