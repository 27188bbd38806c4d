"""Helpers for the GPU parity tests: device transfer and oracle-side references.

Oracle inputs always come from the seeded generators, never from the HIP path.
"""

import sys

import numpy as np
import torch

import oracle
from paper_2608_10010_amd import curvefp as cf

DEV = "cuda:0"
FMTS = ("E4C3", "E5C2", "E3C3", "E4C3_r8/9", "E4C3_r3/4")
BINARY_FMTS = FMTS[:3]


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def to_dev(x: np.ndarray, dtype: str) -> torch.Tensor:
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    if dtype == "bf16":
        t = t.to(torch.bfloat16)       # exact: the generator already rounded to bf16
    return t.to(DEV)


def oracle_quantize(x: np.ndarray, fmt: str, axis: int):
    f = oracle.get_format(fmt)
    if axis == 1:
        return oracle.quantize(x, f)
    return oracle.quantize_axis0(x, f)


def layout_codes(codes: np.ndarray, fmt: str) -> np.ndarray:
    """Oracle codes (one per byte) in the library's storage layout."""
    return oracle.pack7(codes) if fmt == "E3C3" else codes


def unpack_dev_codes(codes: torch.Tensor, fmt: str, k: int) -> np.ndarray:
    c = codes.cpu().numpy()
    if fmt == "E3C3":
        return oracle.unpack7(c.reshape(c.shape[0], -1), k)
    return c


def exact_values(codes: np.ndarray, scales: np.ndarray, fmt: str, block: int = 32) -> np.ndarray:
    """float64 reconstructed values 2^{a + n/K} (the oracle's level function)."""
    f = oracle.get_format(fmt)
    nz, s, n = oracle.code_fields(codes, f)
    a = np.repeat(scales.astype(np.int64), block, axis=1)
    a = np.where(a == oracle.POISON_SCALE, 0, a)
    v = np.ldexp(oracle.level_value_f64(f, np.where(nz, n, 0)), a)
    return np.where(nz, np.where(s == 1, -v, v), 0.0)


def top_exponent(f) -> int:
    """floor(log2) of the format's top level 2^{p n_max / (qK)} (binary radix: 2^{E-1} - 1)."""
    return (f.p * f.n_max) // f.N


def row_tops(codes, scales, fmt):
    """2^{alpha + e_max + 1}: the top of the range a row's block scales allow."""
    f = oracle.get_format(fmt)
    e_max = top_exponent(f)
    sc = scales.astype(np.int64)
    alpha = np.max(np.where(sc == oracle.POISON_SCALE, -127, sc), axis=1)
    return np.ldexp(1.0, alpha + e_max + 1)


# An element is expanded relative to the top of its row's scale range, top = 2^{alpha + e_max + 1}
# (alpha = the row's largest block scale): it keeps 22 significant bits while it stays above
# fp16's normal range in those units, and otherwise an absolute error of at most about 2^-39 top
# (elements below about 2^-41 top are flushed to zero).  FLUSH_REL is that absolute bound with a
# factor of two to spare.
FLUSH_REL = 2.0 ** -38


def element_loss(v: np.ndarray, tops: np.ndarray) -> np.ndarray:
    """Per-element bound on what the expansion can lose beyond the relative 2^-21: at most the
    element itself, and at most FLUSH_REL of its row's top."""
    return np.minimum(v, FLUSH_REL * tops[:, None])


def gemm_tolerance(ca, sa, cb, sb, fmt, block: int = 32):
    """Element-wise bound for the MFMA GEMM against the exact sum.

    * 1e-5 sum_k |a_ik b_jk| covers the 22-bit fp16 high/low operand splits
      (about 3 * 2^-22 per product) and fp32 accumulation;
    * sum_k (la_ik |b_jk| + |a_ik| lb_jk + la_ik lb_jk), with la = element_loss(|a|) (and lb
      for B), covers the elements that fall below fp16's normal range relative to their row's
      top: each such element may lose at most itself and at most 2^-38 of its row's top, so
      the term admits the loss of exactly those contributions and no more;
    * 2^-148 covers an exact result that underflows fp32.
    """
    va, vb = np.abs(exact_values(ca, sa, fmt, block)), np.abs(exact_values(cb, sb, fmt, block))
    la, lb = element_loss(va, row_tops(ca, sa, fmt)), element_loss(vb, row_tops(cb, sb, fmt))
    S = va @ vb.T
    loss = la @ vb.T + va @ lb.T + la @ lb.T
    return 1e-5 * S + loss + 2.0 ** -148


def check_gemm(C_dev: np.ndarray, V: np.ndarray, tol: np.ndarray, what: str, frobenius: bool = True):
    """Element-wise bound `tol` everywhere; relative Frobenius error <= 1e-5 (the workloads'
    bar) unless `frobenius` is off: with K far beyond the workloads' lengths and terms that
    cancel, fp32 accumulation alone can exceed 1e-5 of |C| while staying inside the
    element-wise bound, which scales with sum |a b|."""
    # NaN outputs (rows or columns holding a block that held a NaN or an infinity) must sit
    # exactly where the oracle has them; the bound applies to the rest
    nan_c, nan_v = np.isnan(C_dev), np.isnan(V)
    assert np.array_equal(nan_c, nan_v), f"{what}: NaN at {np.sum(nan_c & ~nan_v)} extra and " \
                                         f"{np.sum(nan_v & ~nan_c)} missing places"
    C64 = np.where(nan_v, 0.0, C_dev.astype(np.float64))
    V = np.where(nan_v, 0.0, V)
    tol = np.where(nan_v, 0.0, tol)
    err = np.abs(C64 - V)
    bad = err > tol
    assert not bad.any(), f"{what}: {bad.sum()} elements beyond bound; worst {np.max(err - tol)}"
    nv = np.linalg.norm(V)
    if nv > 0:
        rel = np.linalg.norm(C64 - V) / nv
        if frobenius:
            assert rel <= 1e-5, f"{what}: relative Frobenius error {rel}"
        return rel
    return 0.0


# ---------------------------------------------------------------- mixed formats, per-element scales

def exact_values_elem(codes: np.ndarray, scales: np.ndarray, fmt: str) -> np.ndarray:
    """float64 values 2^{a + n/K} of codes [R][K] with per-element scales [R][K]."""
    f = oracle.get_format(fmt)
    nz, s, n = oracle.code_fields(codes, f)
    a = scales.astype(np.int64)
    a = np.where(a == oracle.POISON_SCALE, 0, a)
    v = np.ldexp(oracle.level_value_f64(f, np.where(nz, n, 0)), a)
    return np.where(nz, np.where(s == 1, -v, v), 0.0)


def row_tops_elem(scales: np.ndarray, fmt: str) -> np.ndarray:
    f = oracle.get_format(fmt)
    e_max = top_exponent(f)
    sc = scales.astype(np.int64)
    alpha = np.max(np.where(sc == oracle.POISON_SCALE, -127, sc), axis=1)
    return np.ldexp(1.0, alpha + e_max + 1)


def gemm_tolerance_mixed(ca, sa, fa, cb, sb, fb):
    """gemm_tolerance for operands of two formats with per-element scales: each operand's
    elements are expanded relative to the top of its own row's scale range, with its own
    format's largest exponent."""
    va, vb = np.abs(exact_values_elem(ca, sa, fa)), np.abs(exact_values_elem(cb, sb, fb))
    la, lb = element_loss(va, row_tops_elem(sa, fa)), element_loss(vb, row_tops_elem(sb, fb))
    S = va @ vb.T
    loss = la @ vb.T + va @ lb.T + la @ lb.T
    return 1e-5 * S + loss + 2.0 ** -148
