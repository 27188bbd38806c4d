"""Exact CurveFP GEMM (oracle; test infrastructure only).

C[i, j] = sum_k x_hat(A[i, k]) * x_hat(B[j, k])  -- the paper's forward contract
Q_A(X) Q_W(W)^T (Sec. 3.3, App. A.2) with both operands stored K-contiguous.

Two implementations, sharing nothing but the definition:

* ``gemm_exact``: the C library ``curvefp_oracle.c`` -- code-domain products
  accumulated in integer phase bins A[h][t] (Sec. 3.2, App. A.1), exact per-phase
  sums, one rounding in the final fixed-coefficient phase reduction.
* ``gemm_exact_python``: pure Python for tiny cases -- the same bin addressing
  written with Python integers and the phase weights from mpmath.
"""

import ctypes
import os
import subprocess
from fractions import Fraction
from math import gcd

import numpy as np

from .formats import Format
from .quant import POISON_SCALE, code_fields

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "curvefp_oracle.c")
_BUILD_DIR = os.path.join(_HERE, "_build")
_LIB_PATH = os.path.join(_BUILD_DIR, "libcurvefp_oracle.so")
_lib = None


def build_library(force: bool = True) -> str:
    """Compile the C oracle with gcc (host only)."""
    os.makedirs(_BUILD_DIR, exist_ok=True)
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp"
        cmd = ["gcc", "-O2", "-std=gnu11", "-fPIC", "-shared", "-fopenmp", _SRC,
               "-o", tmp, "-lquadmath", "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def load_library():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build_library(force=False)
        lib = ctypes.CDLL(_LIB_PATH)
        P = ctypes.c_void_p
        I64 = ctypes.c_int64
        I = ctypes.c_int
        lib.oracle_gemm_exact.argtypes = [P, P, P, P, I64, I64, I64, I, I, I, I, I, P, I, P]
        lib.oracle_gemm_exact.restype = I
        lib.oracle_dot_phase_sums.argtypes = [P, P, P, P, I64, I, I, I, I, I, P, P, P]
        lib.oracle_dot_phase_sums.restype = I
        lib.oracle_gemm_exact_mixed.argtypes = [P, P, I, I, I, I, P, P, I, I, I, I, I64, I64, I64, P, I, P]
        lib.oracle_gemm_exact_mixed.restype = I
        lib.oracle_max_threads.restype = I
        _lib = lib
    return _lib


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def gemm_exact(a_codes, a_scales, b_codes, b_scales, fmt: Format, block: int = 32,
               nthreads: int = 0, return_max_count: bool = False):
    """Exact GEMM of unpacked codes: A [M, K] x B [N, K]^T -> float64 [M, N]."""
    lib = load_library()
    a_codes = np.ascontiguousarray(a_codes, dtype=np.uint8)
    b_codes = np.ascontiguousarray(b_codes, dtype=np.uint8)
    a_scales = np.ascontiguousarray(a_scales, dtype=np.int8)
    b_scales = np.ascontiguousarray(b_scales, dtype=np.int8)
    M, kd = a_codes.shape
    N, kd2 = b_codes.shape
    assert kd == kd2 and kd % block == 0
    assert a_scales.shape == (M, kd // block) and b_scales.shape == (N, kd // block)
    out = np.empty((M, N), dtype=np.float64)
    mc = np.zeros(1, dtype=np.int32)
    rc = lib.oracle_gemm_exact(_ptr(a_codes), _ptr(a_scales), _ptr(b_codes), _ptr(b_scales),
                               M, N, kd, block, fmt.E, fmt.C, fmt.p, fmt.q,
                               _ptr(out), int(nthreads), _ptr(mc))
    if rc != 0:
        raise ValueError("oracle_gemm_exact rejected its arguments")
    poison_rows_cols(out, a_scales, b_scales)
    if return_max_count:
        return out, int(mc[0])
    return out


def poison_rows_cols(out, a_scales, b_scales):
    """C = deq(A) deq(B)^T where a block that held a NaN or an infinity reconstructs to NaN
    (scale POISON_SCALE, Eq. curvefp-value with the non-finite reading): in IEEE arithmetic
    every dot product that meets a NaN is NaN, zero partners included, so each row of A and
    each row of B with a poisoned scale makes its whole row / column of C NaN."""
    pa = np.any(np.asarray(a_scales) == POISON_SCALE, axis=1)
    pb = np.any(np.asarray(b_scales) == POISON_SCALE, axis=1)
    out[pa, :] = np.nan
    out[:, pb] = np.nan
    return out


def mixed_lattice(fmt_a: Format, fmt_b: Format):
    """Common lattice of two formats: magnitudes 2^(p n / N) of both are integers u over
    D = lcm(N_a, N_b), u_x = p_x (D / N_x) n_x.  Returns (D, la, lb, g, H) with g the gcd of
    the multipliers and D, and H = D / g phases."""
    D = fmt_a.N * fmt_b.N // gcd(fmt_a.N, fmt_b.N)
    la = fmt_a.p * (D // fmt_a.N)
    lb = fmt_b.p * (D // fmt_b.N)
    g = gcd(gcd(la, lb), D)
    return D, la, lb, g, D // g


def gemm_exact_mixed(a_codes, a_scales, fmt_a: Format, b_codes, b_scales, fmt_b: Format,
                     nthreads: int = 0, return_max_count: bool = False):
    """Exact GEMM of two operands in different formats (the backward recipe of Sec. 3.3),
    per-element scales: A codes/scales [M, K], B codes/scales [N, K] -> float64 [M, N].
    Both exponents are taken over the common lattice D = lcm(N_a, N_b) and products are binned
    at h = (u mod D) / g, t = a_x + a_w + floor(u / D) (see curvefp_oracle.c); for binary
    radices D = max(K_a, K_b)."""
    lib = load_library()
    a_codes = np.ascontiguousarray(a_codes, dtype=np.uint8)
    b_codes = np.ascontiguousarray(b_codes, dtype=np.uint8)
    a_scales = np.ascontiguousarray(a_scales, dtype=np.int8)
    b_scales = np.ascontiguousarray(b_scales, dtype=np.int8)
    M, kd = a_codes.shape
    N, kd2 = b_codes.shape
    assert kd == kd2 and a_scales.shape == (M, kd) and b_scales.shape == (N, kd)
    out = np.empty((M, N), dtype=np.float64)
    mc = np.zeros(1, dtype=np.int32)
    rc = lib.oracle_gemm_exact_mixed(_ptr(a_codes), _ptr(a_scales), fmt_a.E, fmt_a.C, fmt_a.p, fmt_a.q,
                                     _ptr(b_codes), _ptr(b_scales), fmt_b.E, fmt_b.C, fmt_b.p, fmt_b.q,
                                     M, N, kd, _ptr(out), int(nthreads), _ptr(mc))
    if rc != 0:
        raise ValueError("oracle_gemm_exact_mixed rejected its arguments")
    poison_rows_cols(out, a_scales, b_scales)
    if return_max_count:
        return out, int(mc[0])
    return out


def expand_scales(scales, block: int = 32, axis: int = 1):
    """Per-element scales from block scales: axis 1 repeats each scale `block` times along
    the last axis (blocks along k); axis 0 takes scales of the transposed operand,
    [k][rows / block], and returns them as [rows][k] (blocks along the rows)."""
    s = np.asarray(scales, dtype=np.int8)
    if axis == 1:
        return np.repeat(s, block, axis=1)
    return np.ascontiguousarray(np.repeat(s, block, axis=1).T)


def product_address_mixed(code_x: int, a_x: int, fmt_x: Format, code_w: int, a_w: int, fmt_w: Format):
    """(delta, h, t) of one product of two formats on their common lattice (mixed_lattice),
    or None for a zero operand."""
    D, lx, lw, g, _ = mixed_lattice(fmt_x, fmt_w)
    ex, ew = fmt_x.E + fmt_x.C, fmt_w.E + fmt_w.C
    mx, mw = code_x & ((1 << ex) - 1), code_w & ((1 << ew) - 1)
    if mx == 0 or mw == 0:
        return None
    sx, sw = (code_x >> ex) & 1, (code_w >> ew) & 1
    u = lx * (mx - fmt_x.B) + lw * (mw - fmt_w.B)
    return (-1 if (sx ^ sw) else 1), (u % D) // g, a_x + a_w + u // D


def phase_bins_one(a_codes, a_scales, b_codes, b_scales, fmt: Format, block: int = 32):
    """One dot product through the C bins: (phase sums N_h [H], value, max |A[h][t]|)."""
    lib = load_library()
    a_codes = np.ascontiguousarray(a_codes, dtype=np.uint8).ravel()
    b_codes = np.ascontiguousarray(b_codes, dtype=np.uint8).ravel()
    a_scales = np.ascontiguousarray(a_scales, dtype=np.int8).ravel()
    b_scales = np.ascontiguousarray(b_scales, dtype=np.int8).ravel()
    kd = a_codes.size
    ph = np.zeros(fmt.H, dtype=np.float64)
    val = np.zeros(1, dtype=np.float64)
    mc = np.zeros(1, dtype=np.int32)
    rc = lib.oracle_dot_phase_sums(_ptr(a_codes), _ptr(a_scales), _ptr(b_codes), _ptr(b_scales),
                                   kd, block, fmt.E, fmt.C, fmt.p, fmt.q,
                                   _ptr(ph), _ptr(val), _ptr(mc))
    if rc != 0:
        raise ValueError("oracle_dot_phase_sums rejected its arguments")
    return ph, float(val[0]), int(mc[0])


def product_address(code_x: int, a_x: int, code_w: int, a_w: int, fmt: Format):
    """(delta, h, t) of one closed product, or None for a zero operand (App. A.1).

    u = p (n_x + n_w), delta = (-1)^(s_x xor s_w), h = (u mod qK) / g,
    t = a_x + a_w + floor(u / qK).
    """
    ec = fmt.E + fmt.C
    mask = (1 << ec) - 1
    mx, mw = code_x & mask, code_w & mask
    if mx == 0 or mw == 0:
        return None
    sx, sw = (code_x >> ec) & 1, (code_w >> ec) & 1
    nx, nw = mx - fmt.B, mw - fmt.B
    N = fmt.N
    u = fmt.p * (nx + nw)
    delta = -1 if (sx ^ sw) else 1
    return delta, (u % N) // fmt.g, a_x + a_w + u // N


def gemm_exact_python(a_codes, a_scales, b_codes, b_scales, fmt: Format, block: int = 32,
                      dps: int = 60):
    """Pure-Python exact GEMM for tiny shapes.

    Counts are kept per (h, t) in a dict, N_h = sum_t count * 2^t is an exact
    Fraction, and V = sum_h 2^(h/H) N_h is evaluated with mpmath at ``dps``
    decimal digits.  Returns float64 [M, N].
    """
    import mpmath

    mpmath.mp.dps = dps
    a_codes = np.asarray(a_codes)
    b_codes = np.asarray(b_codes)
    M, kd = a_codes.shape
    N = b_codes.shape[0]
    weights = [mpmath.power(2, mpmath.mpf(h) / fmt.H) for h in range(fmt.H)]
    out = np.zeros((M, N))
    for i in range(M):
        for j in range(N):
            bins = {}
            for k in range(kd):
                addr = product_address(int(a_codes[i, k]), int(a_scales[i, k // block]),
                                       int(b_codes[j, k]), int(b_scales[j, k // block]), fmt)
                if addr is None:
                    continue
                d, h, t = addr
                bins[(h, t)] = bins.get((h, t), 0) + d
            v = mpmath.mpf(0)
            for h in range(fmt.H):
                nh = sum((Fraction(c) * (Fraction(2) ** t) for (hh, t), c in bins.items() if hh == h),
                         Fraction(0))
                v += weights[h] * mpmath.mpf(nh.numerator) / nh.denominator
            out[i, j] = float(v)
    blocks_a = np.asarray(a_scales)[:, : kd // block]
    blocks_b = np.asarray(b_scales)[:, : kd // block]
    return poison_rows_cols(out, blocks_a, blocks_b)
