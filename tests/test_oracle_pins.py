"""Pins of the CPU oracle against what the paper and the mathematics fix.

CPU only.  Every check here uses a route independent of the code it checks:
paper-printed values (tests/golden/paper_tables.json), rigorous integer
brackets (tests/exact_ref.py), mpmath, exact rationals, or numpy float64
matmul of reconstructed values.
"""

import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle
from oracle import formats as F
from tests import exact_ref as X

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_tables.json")))
FMT_NAMES = ("E4C3", "E5C2", "E3C3")
RADIX_NAMES = ("E4C3_r8/9", "E4C3_r3/4")      # Tab. radix-frontier
ALL_NAMES = FMT_NAMES + RADIX_NAMES


# ------------------------------------------------------------------ tables

@pytest.mark.parametrize("name", FMT_NAMES)
def test_format_table(name):
    """Tab. curvefp-formats: bits, E, C, positive levels and H."""
    g = GOLD["formats"][name]
    f = oracle.get_format(name)
    assert (f.bits, f.E, f.C, f.positive_levels, f.H) == (g["bits"], g["E"], g["C"], g["positive"], g["H"])
    # every canonical magnitude is a distinct level and the codes use exactly bits
    ranks = np.arange(1, 2 ** (f.E + f.C))
    nz, s, n = oracle.code_fields(ranks, f)
    assert nz.all() and len(set(n.tolist())) == g["positive"]
    assert (2 ** (f.E + f.C + 1) - 1) < 2 ** g["bits"]


def test_e5c2_moves_one_bit():
    """Sec. 3.3: E4C3 -> E5C2 keeps 127 levels, phases 8 -> 4."""
    g = GOLD["e5c2_vs_e4c3"]
    a, b = oracle.get_format("E4C3"), oracle.get_format("E5C2")
    assert a.positive_levels == b.positive_levels == g["levels"]
    assert (a.H, b.H) == (g["H_from"], g["H_to"])


def _occupied_phases(f):
    """Phases actually hit by all nonzero code pairs (brute force over the codebook)."""
    seen = set()
    mags = range(1, 2 ** (f.E + f.C))
    for mx in mags:
        for mw in mags:
            d, h, t = oracle.product_address(mx, 0, mw, 0, f)
            seen.add(h)
    return seen


@pytest.mark.parametrize("case", GOLD["radix_phases"]["cases"], ids=lambda c: f"p{c['p']}q{c['q']}")
def test_phase_count_rational_radix(case):
    """Tab. radix-frontier: 8 / 9 / 32 phases; brute-force occupancy equals H."""
    f = oracle.rational_format(case["E"], case["C"], case["p"], case["q"])
    assert f.H == case["H"]
    assert _occupied_phases(f) == set(range(case["H"]))


@pytest.mark.parametrize("name", FMT_NAMES)
def test_phase_count_principal(name):
    f = oracle.get_format(name)
    assert _occupied_phases(f) == set(range(GOLD["formats"][name]["H"]))


def test_storage_rates():
    """Sec. 4.2 / Eq. effective-rate: printed E3C3 rates are met with integer S."""
    f = oracle.get_format(GOLD["storage_rates"]["format"])
    for c in GOLD["storage_rates"]["cases"]:
        ok = [S for S in range(1, 9) if round(f.storage_rate(c["G"], S), 3) == c["printed"]]
        assert ok, c


def test_e4c3_tile_encoding():
    """App. C.1: q = m - 64 and q_p = m_a + m_b - 128 = 8e + k for every pair."""
    g = GOLD["tile_encoding"]
    f = oracle.get_format("E4C3")
    for ma in range(1, 128):
        for sa in (0, 1):
            code_a = (sa << g["sign_bit"]) | ma
            nz, s, n = (int(v[0]) for v in oracle.code_fields(np.array([code_a]), f))
            assert nz and s == sa and n == ma - g["q_offset"]
    for ma in range(1, 128):
        for mb in range(1, 128):
            d, h, t = oracle.product_address(ma, 0, mb | 0x80, 0, f)
            qp = ma + mb - g["product_offset"]
            e, k = divmod(qp, g["curves"])
            assert (h, t, d) == (k, e, -1)


# ------------------------------------------------------------------ closure

@pytest.mark.parametrize("name", FMT_NAMES)
def test_closed_product_all_pairs(name):
    """Eq. curve-index-product vs the bin address of App. A.1, and the value.

    For every pair of nonzero codes (both signs) and a few scale pairs:
    l = (i + j) mod K, c = floor((i + j) / K), exponent e_x + e_w + c and sign
    xor must equal (h, t, delta) of the general addressing, and
    delta 2^t 2^(h/H) must equal the product of the two reconstructed values
    computed from their (s, e, k) fields with mpmath.
    """
    import mpmath
    mpmath.mp.dps = 40
    f = oracle.get_format(name)
    K = f.K
    mags = np.arange(1, 2 ** (f.E + f.C))
    codes = np.concatenate([mags, mags | (1 << (f.E + f.C))])
    nz, s, n = oracle.code_fields(codes, f)
    e, k = np.floor_divide(n, K), np.mod(n, K)
    rng = np.random.default_rng(0)
    scale_pairs = [(0, 0), (-5, 3)]
    for ax, aw in scale_pairs:
        for ix in range(len(codes)):
            for iw in range(len(codes)):
                d, h, t = oracle.product_address(int(codes[ix]), ax, int(codes[iw]), aw, f)
                l = (k[ix] + k[iw]) % K
                c = (k[ix] + k[iw]) // K
                assert h == l
                assert t == ax + aw + e[ix] + e[iw] + c
                assert d == (-1 if s[ix] ^ s[iw] else 1)
        # numeric value on a random subset (mpmath is slow)
        for _ in range(300):
            ix, iw = rng.integers(0, len(codes), 2)
            d, h, t = oracle.product_address(int(codes[ix]), ax, int(codes[iw]), aw, f)
            vx = (-1) ** int(s[ix]) * mpmath.power(2, ax) * mpmath.power(2, int(e[ix]) + mpmath.mpf(int(k[ix])) / K)
            vw = (-1) ** int(s[iw]) * mpmath.power(2, aw) * mpmath.power(2, int(e[iw]) + mpmath.mpf(int(k[iw])) / K)
            got = d * mpmath.power(2, t) * mpmath.power(2, mpmath.mpf(h) / f.H)
            assert abs(got - vx * vw) <= mpmath.mpf(10) ** -30 * abs(vx * vw)


def test_zero_short_circuits():
    f = oracle.get_format("E4C3")
    for c in (0x00, 0x80):
        assert oracle.product_address(c, 0, 0x45, 0, f) is None
        assert oracle.product_address(0x45, 0, c, 0, f) is None


# ------------------------------------------------------------------ quantizer

def _blocks_with_scale0(values, f):
    """Blocks of 32 whose first element is fl32(L_max), so the block scale is 0."""
    lm = np.float32(oracle.level_value_f64(f, f.n_max))
    per = 31
    nb = -(-len(values) // per)
    buf = np.zeros(nb * per, np.float32)
    buf[: len(values)] = values
    blocks = np.concatenate([np.full((nb, 1), lm, np.float32), buf.reshape(nb, per)], axis=1)
    return blocks.reshape(1, -1), nb


def _rigorous_codes(Ms, j, f):
    out = []
    for M in Ms:
        n = X.nearest_binary_radix(int(M), j, f.E, f.C)
        out.append(0 if n is None else n + f.B)
    return np.array(out)


@pytest.mark.parametrize("name", FMT_NAMES)
def test_nearest_level_exhaustive_octave(name):
    """Every fp32 significand of an interior octave: oracle == rigorous decision.

    The rigorous decision brackets each midpoint (2^(c/K) + 2^((c+1)/K)) / 2 with
    integer K-th roots.  Decisions only depend on the significand within an
    octave (the rule is the same in every octave), so this covers every
    interior element exactly.
    """
    f = oracle.get_format(name)
    j = 0
    Ms = np.arange(1 << 23, 1 << 24, dtype=np.int64)
    vals = np.ldexp(Ms.astype(np.float64), j - 23).astype(np.float32)
    x, nb = _blocks_with_scale0(vals, f)
    codes, scales = oracle.quantize(x, f)
    assert np.all(scales == 0)
    got = codes.reshape(nb, 32)[:, 1:].reshape(-1)[: len(Ms)].astype(np.int64)
    # rigorous thresholds: the decision changes only at K integer thresholds
    K = f.K
    thr = []
    for c in range(K):
        lo, hi = (1 << 23), (1 << 24) - 1
        # find the largest M that is NOT above threshold c (binary search on the rigorous rule)
        def above(M):
            n = X.nearest_binary_radix(M, j, f.E, f.C)
            return n is not None and n - K * j > c
        while lo < hi:
            mid = (lo + hi + 1) // 2
            if above(mid):
                hi = mid - 1
            else:
                lo = mid
        thr.append(lo)
    expect_c = np.zeros(len(Ms), np.int64)
    for t in thr:
        expect_c += (Ms > t)
    expect = K * j + expect_c + f.B
    assert np.array_equal(got, expect)
    # spot-check the rigorous rule itself on the neighbours of each threshold
    for t in thr:
        for M in (t - 1, t, t + 1, t + 2):
            if (1 << 23) <= M < (1 << 24):
                assert _rigorous_codes([M], j, f)[0] == expect[M - (1 << 23)]


@pytest.mark.parametrize("name", FMT_NAMES)
def test_nearest_level_edges(name):
    """Octaves around the zero threshold, the smallest level and the top level."""
    f = oracle.get_format(name)
    rng = np.random.default_rng(1)
    e_min = math.floor(f.n_min / f.K)
    e_max = math.floor(f.n_max / f.K)
    for j in (e_min - 3, e_min - 2, e_min - 1, e_min, e_min + 1, e_max):
        Ms = np.unique(np.concatenate([
            rng.integers(1 << 23, 1 << 24, 20000),
            np.array([1 << 23, (1 << 24) - 1]),
        ]))
        vals = np.ldexp(Ms.astype(np.float64), j - 23).astype(np.float32)
        # values above fl32(L_max) would raise the block scale; they are not in scope here
        lm = float(np.float32(oracle.level_value_f64(f, f.n_max)))
        keep = vals.astype(np.float64) <= lm
        Ms, vals = Ms[keep], vals[keep]
        x, nb = _blocks_with_scale0(vals, f)
        codes, scales = oracle.quantize(x, f)
        assert np.all(scales == 0)
        got = codes.reshape(nb, 32)[:, 1:].reshape(-1)[: len(Ms)].astype(np.int64)
        exp = _rigorous_codes(Ms, j, f)
        assert np.array_equal(got, exp), j


@pytest.mark.parametrize("name", FMT_NAMES)
def test_scale_rule_and_error_bound(name):
    """Ceil-absmax: the block max lands in (fl32(L_max)/2, fl32(L_max)] after scaling,
    and interior elements obey |x - x_hat| <= |x| (2^(1/K) - 1) / (2^(1/K) + 1)."""
    f = oracle.get_format(name)
    rng = np.random.default_rng(2)
    x = (rng.standard_normal((64, 1024)) * np.exp2(rng.uniform(-30, 30, (64, 1)))).astype(np.float32)
    codes, scales = oracle.quantize(x, f)
    lm = float(np.float32(oracle.level_value_f64(f, f.n_max)))
    amax = np.abs(x.astype(np.float64)).reshape(64, 32, 32).max(-1)
    y = np.ldexp(amax, -scales.astype(np.int64))
    assert np.all(y <= lm) and np.all(y > lm / 2)
    deq = oracle.dequantize(codes, scales, f).astype(np.float64)
    xd = x.astype(np.float64)
    bound = (2 ** (1 / f.K) - 1) / (2 ** (1 / f.K) + 1)
    a = np.repeat(scales.astype(np.int64), 32, axis=1)
    interior = (np.abs(xd) >= np.ldexp(oracle.level_value_f64(f, f.n_min), a))
    rel = np.abs(xd - deq)[interior] / np.abs(xd)[interior]
    assert rel.max() <= bound * (1 + 1e-6)
    # saturation never fires under this scale rule: no element beyond the top level
    nz, s, n = oracle.code_fields(codes, f)
    assert np.all(n[nz] <= f.n_max)


@pytest.mark.parametrize("name", ALL_NAMES)
@pytest.mark.parametrize("a", [-100, -20, 0, 7, 100])
def test_round_trip_all_codes(name, a):
    """quantize(dequantize(c)) == c for every canonical code (blocks holding the top code)."""
    f = oracle.get_format(name)
    EC = f.E + f.C
    mags = np.arange(1, 2 ** EC)
    allc = np.concatenate([mags, mags | (1 << EC)]).astype(np.uint8)
    top = np.uint8(2 ** EC - 1)
    per = 31
    nb = -(-len(allc) // per)
    body = np.zeros(nb * per, np.uint8)
    body[: len(allc)] = allc
    codes = np.concatenate([np.full((nb, 1), top, np.uint8), body.reshape(nb, per)], axis=1).reshape(1, -1)
    scales = np.full((1, nb), a, np.int8)
    deq = oracle.dequantize(codes, scales, f)
    c2, s2 = oracle.quantize(deq, f)
    assert np.array_equal(s2, scales)
    assert np.array_equal(c2, codes)


@pytest.mark.parametrize("name", FMT_NAMES)
def test_dequantize_rigorous_all_codes_all_scales(name):
    """fp32 reconstruction == rigorously rounded 2^(a + n/K), every code and scale."""
    f = oracle.get_format(name)
    EC = f.E + f.C
    mags = np.arange(1, 2 ** EC)
    scales = np.arange(-127, 128)
    codes = np.tile(mags, (len(scales), 1)).astype(np.uint8)
    codes = np.repeat(codes, 1, axis=1)
    # one block per (scale, 32 codes): lay codes out so each block has one scale
    nmag = len(mags)
    pad = (-nmag) % 32
    cpad = np.concatenate([codes, np.zeros((len(scales), pad), np.uint8)], axis=1)
    sc = np.repeat(scales[:, None], cpad.shape[1] // 32, axis=1).astype(np.int8)
    got = oracle.dequantize(cpad, sc, f)[:, :nmag]
    for ia, a in enumerate(scales):
        for im, m in enumerate(mags):
            exp = X.rn_f32_pow2(int(a), int(m) - f.B, f.K)
            g = float(got[ia, im])
            assert X.f32_bits(g) == X.f32_bits(exp), (a, m, g, exp)
    neg = oracle.dequantize(cpad | np.uint8(1 << EC), sc, f)[:, :nmag]
    assert np.array_equal(neg, -got)
    zero = oracle.dequantize(np.zeros_like(cpad), sc, f)
    assert np.all(zero == 0) and not np.any(np.signbit(zero))


def test_nonfinite_blocks_poison():
    f = oracle.get_format("E4C3")
    x = np.ones((2, 64), np.float32)
    x[0, 3] = np.nan
    x[1, 40] = -np.inf
    codes, scales = oracle.quantize(x, f)
    assert scales[0, 0] == oracle.POISON_SCALE and scales[1, 1] == oracle.POISON_SCALE
    assert scales[0, 1] != oracle.POISON_SCALE and scales[1, 0] != oracle.POISON_SCALE
    assert np.all(codes[0, :32] == 0) and np.all(codes[1, 32:] == 0)
    d = oracle.dequantize(codes, scales, f)
    assert np.all(np.isnan(d[0, :32])) and np.all(np.isnan(d[1, 32:]))


def test_zero_block_and_sign_of_zero():
    """All-zero blocks (either sign of zero) give code 0 and the bottom scale -127: for a zero
    maximum every integer a satisfies the ceil-absmax inequality, and -127 is the smallest stored
    scale.  A block whose maximum is the smallest subnormal lands on the same scale."""
    f = oracle.get_format("E5C2")
    x = np.zeros((1, 96), np.float32)
    x[0, 32:64] = -0.0
    x[0, 64] = np.float32(2.0 ** -149)
    codes, scales = oracle.quantize(x, f)
    assert np.all(codes[0, :64] == 0) and np.all(scales == -127)


def test_pack7_layout():
    """7-bit packing: code i at bits [7i, 7i+7) of a 224-bit little-endian string."""
    rng = np.random.default_rng(3)
    codes = rng.integers(0, 128, (5, 96)).astype(np.uint8)
    packed = oracle.pack7(codes)
    assert packed.shape == (5, 3, 28)
    for r in range(5):
        for b in range(3):
            big = sum(int(c) << (7 * i) for i, c in enumerate(codes[r, 32 * b: 32 * b + 32]))
            assert bytes(packed[r, b]) == big.to_bytes(28, "little")
    assert np.array_equal(oracle.unpack7(packed, 96), codes)


# ------------------------------------------------------------------ GEMM

def _deq_exact64(codes, scales, f):
    nz, s, n = oracle.code_fields(codes, f)
    a = np.repeat(scales.astype(np.int64), 32, axis=1)
    v = np.ldexp(oracle.level_value_f64(f, np.where(nz, n, 0)), a)
    return np.where(nz, np.where(s == 1, -v, v), 0.0)


@pytest.mark.parametrize("name", ALL_NAMES)
def test_gemm_matches_float64_matmul(name):
    """Phase-binned exact GEMM vs numpy float64 matmul of reconstructed values."""
    f = oracle.get_format(name)
    rng = np.random.default_rng(4)
    A = (rng.standard_normal((48, 256)) * np.exp2(rng.uniform(-8, 8, (48, 1)))).astype(np.float32)
    B = (rng.standard_normal((40, 256)) * 0.02).astype(np.float32)
    ca, sa = oracle.quantize(A, f)
    cb, sb = oracle.quantize(B, f)
    C = oracle.gemm_exact(ca, sa, cb, sb, f)
    ref = _deq_exact64(ca, sa, f) @ _deq_exact64(cb, sb, f).T
    absmm = np.abs(_deq_exact64(ca, sa, f)) @ np.abs(_deq_exact64(cb, sb, f)).T
    assert np.all(np.abs(C - ref) <= 1e-13 * absmm)
    # transposed operands would not even have the right shape or values
    assert C.shape == (48, 40)


@pytest.mark.parametrize("name", ALL_NAMES)
def test_gemm_matches_python_mini_oracle(name):
    f = oracle.get_format(name)
    rng = np.random.default_rng(5)
    A = rng.standard_normal((3, 64)).astype(np.float32)
    B = rng.standard_normal((4, 64)).astype(np.float32)
    ca, sa = oracle.quantize(A, f)
    cb, sb = oracle.quantize(B, f)
    C = oracle.gemm_exact(ca, sa, cb, sb, f)
    P = oracle.gemm_exact_python(ca, sa, cb, sb, f)
    assert np.allclose(C, P, rtol=1e-15, atol=0)


def test_gemm_powers_of_two_exact():
    """All curve indices zero: every product is +-2^t, so the dot is an exact rational."""
    f = oracle.get_format("E5C2")
    rng = np.random.default_rng(6)
    M, N, K = 4, 5, 96
    e_a = rng.integers(-15, 16, (M, K))   # n = 4e >= n_min = -63
    e_b = rng.integers(-15, 16, (N, K))
    ca = ((rng.integers(0, 2, (M, K)) << 7) | (e_a * f.K + f.B)).astype(np.uint8)
    cb = ((rng.integers(0, 2, (N, K)) << 7) | (e_b * f.K + f.B)).astype(np.uint8)
    sa = rng.integers(-100, 100, (M, K // 32)).astype(np.int8)
    sb = rng.integers(-100, 100, (N, K // 32)).astype(np.int8)
    C = oracle.gemm_exact(ca, sa, cb, sb, f)
    for i in range(M):
        for j in range(N):
            tot = Fraction(0)
            for k in range(K):
                sgn = -1 if ((ca[i, k] >> 7) ^ (cb[j, k] >> 7)) & 1 else 1
                ex = int(e_a[i, k] + e_b[j, k] + sa[i, k // 32] + sb[j, k // 32])
                tot += sgn * Fraction(2) ** ex
            assert C[i, j] == float(tot)


@pytest.mark.parametrize("name", ALL_NAMES)
def test_gemm_sign_identity_and_zero(name):
    f = oracle.get_format(name)
    EC = f.E + f.C
    rng = np.random.default_rng(7)
    A = rng.standard_normal((8, 64)).astype(np.float32)
    ca, sa = oracle.quantize(A, f)
    # identity-like B: row j has the level 1.0 (n = 0) at column j, zeros elsewhere
    cb = np.zeros((64, 64), np.uint8)
    cb[np.arange(64), np.arange(64)] = f.B          # m = B  <=> n = 0  <=> value 1 at scale 0
    sb = np.zeros((64, 2), np.int8)
    C = oracle.gemm_exact(ca, sa, cb, sb, f)
    assert np.array_equal(C, _deq_exact64(ca, sa, f))
    neg = np.where(ca != 0, ca ^ np.uint8(1 << EC), 0).astype(np.uint8)
    Cn = oracle.gemm_exact(neg, sa, cb, sb, f)
    assert np.array_equal(Cn, -C)
    Cz = oracle.gemm_exact(np.zeros_like(ca), sa, cb, sb, f)
    assert np.all(Cz == 0)


def test_counter_width_bound():
    """Sec. 3.2: |A[h][t]| <= D, and D fits a 1 + ceil(log2(D+1)) bit signed counter."""
    f = oracle.get_format("E4C3")
    for D in (32, 4096):
        a = np.full(D, 0x55, np.uint8)
        b = np.full(D, 0x41, np.uint8)
        s = np.zeros(D // 32, np.int8)
        ph, val, mc = oracle.phase_bins_one(a, s, b, s, f)
        assert mc == D                       # all products land in one bin: the bound is tight
        width = 1 + math.ceil(math.log2(D + 1))
        assert -(2 ** (width - 1)) <= -D and D <= 2 ** (width - 1) - 1
    assert [1 + math.ceil(math.log2(D + 1)) for D in (32, 4096, 11008, 14336)] == [7, 14, 15, 15]
    # a random dot never exceeds the bound either
    rng = np.random.default_rng(8)
    A = rng.standard_normal((4, 4096)).astype(np.float32)
    ca, sa = oracle.quantize(A, f)
    _, mc = oracle.gemm_exact(ca, sa, ca, sa, f, return_max_count=True)
    assert mc <= 4096


def test_phase_sums_recombine():
    """sum_h 2^(h/H) N_h reproduces the returned value; N_h are integers times 2^t."""
    f = oracle.get_format("E3C3")
    rng = np.random.default_rng(9)
    x = rng.standard_normal((1, 256)).astype(np.float32)
    w = rng.standard_normal((1, 256)).astype(np.float32)
    ca, sa = oracle.quantize(x, f)
    cb, sb = oracle.quantize(w, f)
    ph, val, mc = oracle.phase_bins_one(ca, sa, cb, sb, f)
    assert len(ph) == f.H
    v2 = sum(2 ** (h / f.H) * ph[h] for h in range(f.H))
    assert abs(v2 - val) <= 1e-12 * abs(val)
    ref = (_deq_exact64(ca, sa, f) @ _deq_exact64(cb, sb, f).T)[0, 0]
    assert abs(val - ref) <= 1e-12 * abs(ref)


# ------------------------------------------------------------------ rational radix (Tab. radix-frontier)

def _rigorous_rank(M, j, f):
    n = X.nearest_level(int(M), j, f.E, f.C, f.p, f.q)
    return 0 if n is None else n + f.B


def _rank_steps(j, f):
    """The rigorous rank over the significands of octave j as a step function: [(first M, rank)]."""
    lo_M, hi_M = 1 << 23, (1 << 24) - 1
    steps = [(lo_M, _rigorous_rank(lo_M, j, f))]
    r_end = _rigorous_rank(hi_M, j, f)
    while steps[-1][1] != r_end:
        cur = steps[-1][1]
        lo, hi = steps[-1][0], hi_M
        while lo < hi:                      # smallest M whose rank exceeds cur
            mid = (lo + hi) // 2
            if _rigorous_rank(mid, j, f) > cur:
                hi = mid
            else:
                lo = mid + 1
        steps.append((lo, _rigorous_rank(lo, j, f)))
    return steps


@pytest.mark.parametrize("name", RADIX_NAMES)
def test_radix_format_parameters(name):
    """Tab. radix-frontier variants: E4C3 element (8 bits, 127 positive magnitudes), levels
    2^(p n / (qK)) (Sec. 3.2: r^(e + k/K) = 2^(p(eK + k)/(qK))), H from the printed table."""
    f = oracle.get_format(name)
    case = next(c for c in GOLD["radix_phases"]["cases"] if (c["p"], c["q"]) == (f.p, f.q))
    assert (f.bits, f.E, f.C, f.positive_levels, f.H) == (8, case["E"], case["C"], 127, case["H"])
    n = np.arange(f.n_min, f.n_max + 1)
    v = oracle.level_value_f64(f, n)
    r = 2.0 ** (f.p / f.q)
    assert np.allclose(v, r ** (n / f.K), rtol=1e-14, atol=0)
    assert np.all(np.diff(v) > 0)
    # adjacent curve indices differ by r^(1/K), adjacent exponents by r (Sec. 3.1)
    assert np.allclose(v[1:] / v[:-1], r ** (1 / f.K), rtol=1e-14)
    assert np.allclose(v[f.K:] / v[:-f.K], r, rtol=1e-14)


@pytest.mark.parametrize("name", RADIX_NAMES)
def test_radix_nearest_level_exhaustive_octaves(name):
    """Every fp32 significand of the interior octaves over one period of the level pattern
    (1 octave for 2^(1/9) spacing, 3 for 2^(3/32)): oracle == rigorous nearest level."""
    f = oracle.get_format(name)
    period = f.p // math.gcd(f.p, f.N)
    Ms = np.arange(1 << 23, 1 << 24, dtype=np.int64)
    for j in range(period):
        vals = np.ldexp(Ms.astype(np.float64), j - 23).astype(np.float32)
        x, nb = _blocks_with_scale0(vals, f)
        codes, scales = oracle.quantize(x, f)
        assert np.all(scales == 0)
        got = codes.reshape(nb, 32)[:, 1:].reshape(-1)[: len(Ms)].astype(np.int64)
        steps = _rank_steps(j, f)
        assert len(steps) >= 9                    # at least 9 levels' decisions per octave here
        expect = np.zeros(len(Ms), np.int64)
        for M0, r in steps:
            expect[M0 - (1 << 23):] = r
        assert np.array_equal(got, expect), j


@pytest.mark.parametrize("name", RADIX_NAMES)
def test_radix_nearest_level_edges(name):
    """Octaves around the zero threshold, the smallest level and the top level."""
    f = oracle.get_format(name)
    rng = np.random.default_rng(11)
    w_min = (f.p * f.n_min) // f.N
    w_max = (f.p * f.n_max) // f.N
    lm = float(np.float32(oracle.level_value_f64(f, f.n_max)))
    for j in (w_min - 3, w_min - 2, w_min - 1, w_min, w_min + 1, w_max - 1, w_max):
        Ms = np.unique(np.concatenate([rng.integers(1 << 23, 1 << 24, 3000),
                                       np.array([1 << 23, (1 << 23) + 1, (1 << 24) - 1])]))
        vals = np.ldexp(Ms.astype(np.float64), j - 23).astype(np.float32)
        keep = vals.astype(np.float64) <= lm
        Ms, vals = Ms[keep], vals[keep]
        x, nb = _blocks_with_scale0(vals, f)
        codes, scales = oracle.quantize(x, f)
        assert np.all(scales == 0)
        got = codes.reshape(nb, 32)[:, 1:].reshape(-1)[: len(Ms)].astype(np.int64)
        exp = np.array([_rigorous_rank(M, j, f) for M in Ms])
        assert np.array_equal(got, exp), j


def test_radix_zero_tie_goes_to_the_level():
    """r = 2^(8/9): the smallest level is 2^(-7), so the zero/level decision point 2^(-8) is a
    float and a tie can occur (with binary radix and r = 2^(3/4) it is irrational).  Reading: the
    tie goes to the smallest level; one ulp below goes to zero."""
    f = oracle.get_format("E4C3_r8/9")
    assert oracle.level_value_f64(f, f.n_min) == 2.0 ** -7
    half = np.float32(2.0 ** -8)
    below = np.nextafter(half, np.float32(0))
    x, nb = _blocks_with_scale0(np.array([half, below, -half], np.float32), f)
    codes, scales = oracle.quantize(x, f)
    assert scales[0, 0] == 0
    assert list(codes[0, 1:4]) == [1, 0, 1 | (1 << (f.E + f.C))]
    assert X.nearest_level(1 << 23, -8, f.E, f.C, f.p, f.q) == f.n_min
    for name in ("E4C3", "E4C3_r3/4"):     # elsewhere the point is irrational: no tie
        g = oracle.get_format(name)
        _, r = divmod(g.p * g.n_min, g.N)
        assert r != 0


@pytest.mark.parametrize("name", RADIX_NAMES)
def test_radix_scale_rule_and_error_bound(name):
    """Ceil-absmax with the fp32 top level, and the interior bound |x - x_hat| <= |x| (rho - 1) /
    (rho + 1) for the level ratio rho = r^(1/K)."""
    f = oracle.get_format(name)
    rng = np.random.default_rng(12)
    x = (rng.standard_normal((64, 1024)) * np.exp2(rng.uniform(-30, 30, (64, 1)))).astype(np.float32)
    codes, scales = oracle.quantize(x, f)
    lm = float(np.float32(oracle.level_value_f64(f, f.n_max)))
    amax = np.abs(x.astype(np.float64)).reshape(64, 32, 32).max(-1)
    y = np.ldexp(amax, -scales.astype(np.int64))
    assert np.all(y <= lm) and np.all(y > lm / 2)
    deq = oracle.dequantize(codes, scales, f).astype(np.float64)
    xd = x.astype(np.float64)
    rho = 2.0 ** (f.p / f.N)
    bound = (rho - 1) / (rho + 1)
    a = np.repeat(scales.astype(np.int64), 32, axis=1)
    interior = np.abs(xd) >= np.ldexp(oracle.level_value_f64(f, f.n_min), a)
    rel = np.abs(xd - deq)[interior] / np.abs(xd)[interior]
    assert rel.max() <= bound * (1 + 1e-6)
    nz, s, n = oracle.code_fields(codes, f)
    assert np.all(n[nz] <= f.n_max)


@pytest.mark.parametrize("name", RADIX_NAMES)
def test_radix_dequantize_rigorous_all_codes_all_scales(name):
    """fp32 reconstruction == rigorously rounded 2^(a + p n / N), every code and scale."""
    f = oracle.get_format(name)
    EC = f.E + f.C
    mags = np.arange(1, 2 ** EC)
    scales = np.arange(-127, 128)
    pad = (-len(mags)) % 32
    cpad = np.concatenate([np.tile(mags, (len(scales), 1)), np.zeros((len(scales), pad), np.int64)],
                          axis=1).astype(np.uint8)
    sc = np.repeat(scales[:, None], cpad.shape[1] // 32, axis=1).astype(np.int8)
    got = oracle.dequantize(cpad, sc, f)[:, :len(mags)]
    for ia, a in enumerate(scales):
        for im, m in enumerate(mags):
            exp = X.rn_f32_level(int(a), int(m) - f.B, f.p, f.N)
            assert X.f32_bits(float(got[ia, im])) == X.f32_bits(exp), (a, m)


@pytest.mark.parametrize("name", RADIX_NAMES)
def test_radix_closed_product_values(name):
    """Closure with a rational radix (Sec. 3.2): every code pair's (delta, h, t) gives
    delta 2^t 2^(h/H) equal to the product of the two reconstructed values (mpmath)."""
    import mpmath
    mpmath.mp.dps = 40
    f = oracle.get_format(name)
    mags = np.arange(1, 2 ** (f.E + f.C))
    r = mpmath.power(2, mpmath.mpf(f.p) / f.q)
    for mx in mags[::3]:
        for mw in mags[::5]:
            d, h, t = oracle.product_address(int(mx), -3, int(mw | (1 << 7)), 5, f)
            got = d * mpmath.power(2, t) * mpmath.power(2, mpmath.mpf(h) / f.H)
            vx = mpmath.power(2, -3) * mpmath.power(r, mpmath.mpf(int(mx) - f.B) / f.K)
            vw = -mpmath.power(2, 5) * mpmath.power(r, mpmath.mpf(int(mw) - f.B) / f.K)
            assert abs(got - vx * vw) <= mpmath.mpf(10) ** -30 * abs(vx * vw)


# ------------------------------------------------------------------ mixed formats (backward recipe)

MIXED = [("E5C2", "E4C3"), ("E4C3", "E5C2"), ("E5C2", "E3C3")]


@pytest.mark.parametrize("pair", MIXED, ids=lambda p: f"{p[0]}x{p[1]}")
def test_mixed_product_closure_all_pairs(pair):
    """Sec. 3.3 training protocol (E5C2 gradients x E4C3 forward operands): every pair of
    nonzero codes of the two formats, both signs, a few scale pairs.  The address on the
    lattice L = max(K_x, K_w) must give delta 2^t 2^(h/L) equal to the product of the two
    values built from their own (s, e, k) fields with mpmath; every one of the L phases is
    occupied."""
    import mpmath
    mpmath.mp.dps = 40
    fx, fw = oracle.get_format(pair[0]), oracle.get_format(pair[1])
    L = max(fx.K, fw.K)

    def fields(f):
        mags = np.arange(1, 2 ** (f.E + f.C))
        codes = np.concatenate([mags, mags | (1 << (f.E + f.C))])
        nz, s, n = oracle.code_fields(codes, f)
        return codes, s, np.floor_divide(n, f.K), np.mod(n, f.K)

    cx, sx, ex, kx = fields(fx)
    cw, sw, ew, kw = fields(fw)
    phases = set()
    rng = np.random.default_rng(11)
    for ax, aw in [(0, 0), (-7, 4)]:
        for i in range(len(cx)):
            for j in range(len(cw)):
                d, h, t = oracle.product_address_mixed(int(cx[i]), ax, fx, int(cw[j]), aw, fw)
                # independent form: exponents and curve fractions added as rationals
                q = Fraction(int(ex[i])) + Fraction(int(kx[i]), fx.K) + Fraction(int(ew[j])) + Fraction(int(kw[j]), fw.K)
                assert Fraction(t - ax - aw) + Fraction(h, L) == q
                assert 0 <= h < L and d == (-1 if sx[i] ^ sw[j] else 1)
                phases.add(h)
        for _ in range(200):
            i, j = int(rng.integers(0, len(cx))), int(rng.integers(0, len(cw)))
            d, h, t = oracle.product_address_mixed(int(cx[i]), ax, fx, int(cw[j]), aw, fw)
            vx = (-1) ** int(sx[i]) * mpmath.power(2, ax + int(ex[i]) + mpmath.mpf(int(kx[i])) / fx.K)
            vw = (-1) ** int(sw[j]) * mpmath.power(2, aw + int(ew[j]) + mpmath.mpf(int(kw[j])) / fw.K)
            got = d * mpmath.power(2, t) * mpmath.power(2, mpmath.mpf(h) / L)
            assert abs(got - vx * vw) <= mpmath.mpf(10) ** -30 * abs(vx * vw)
    assert phases == set(range(L))
    assert oracle.product_address_mixed(0, 0, fx, int(cw[5]), 0, fw) is None
    assert oracle.product_address_mixed(int(cx[5]), 0, fx, 0, 0, fw) is None


def test_mixed_equals_single_format_when_formats_agree():
    """With both operands in one format the lifted rule is the paper's single-format rule:
    the mixed oracle (per-element scales) must reproduce gemm_exact bit for bit."""
    rng = np.random.default_rng(12)
    for name in ALL_NAMES:
        f = oracle.get_format(name)
        A = (rng.standard_normal((9, 96)) * np.exp2(rng.uniform(-5, 5, (9, 1)))).astype(np.float32)
        B = rng.standard_normal((7, 96)).astype(np.float32)
        ca, sa = oracle.quantize(A, f)
        cb, sb = oracle.quantize(B, f)
        C1 = oracle.gemm_exact(ca, sa, cb, sb, f)
        C2 = oracle.gemm_exact_mixed(ca, oracle.expand_scales(sa), f, cb, oracle.expand_scales(sb), f)
        assert np.array_equal(C1, C2)


@pytest.mark.parametrize("pair", MIXED, ids=lambda p: f"{p[0]}x{p[1]}")
def test_mixed_gemm_matches_float64_matmul(pair):
    """Mixed exact GEMM vs numpy float64 matmul of each operand reconstructed in its own
    format (a textbook route that shares no binning logic)."""
    fa, fb = oracle.get_format(pair[0]), oracle.get_format(pair[1])
    rng = np.random.default_rng(13)
    A = (rng.standard_normal((40, 192)) * np.exp(rng.normal(0, 3, (40, 1)))).astype(np.float32)
    B = (rng.standard_normal((36, 192)) * 0.02).astype(np.float32)
    ca, sa = oracle.quantize(A, fa)
    cb, sb = oracle.quantize(B, fb)
    C = oracle.gemm_exact_mixed(ca, oracle.expand_scales(sa), fa, cb, oracle.expand_scales(sb), fb)
    da, db = _deq_exact64(ca, sa, fa), _deq_exact64(cb, sb, fb)
    ref = da @ db.T
    absmm = np.abs(da) @ np.abs(db).T
    assert np.all(np.abs(C - ref) <= 1e-13 * absmm)
    # the single-format oracle in either format is a different product
    assert not np.allclose(oracle.gemm_exact(ca, sa, cb, sb, fa), ref, rtol=1e-6, atol=0)


def test_mixed_gemm_with_reused_forward_codes():
    """The backward GEMMs reuse forward codes whose blocks lie along the non-contraction axis
    (dgrad: W [d_out, d_in] blocked along d_in, contracted over d_out).  B is given as the
    codes of B^T quantized along B's rows; per-element scales follow the other axis."""
    fg, fw = oracle.get_format("E5C2"), oracle.get_format("E4C3")
    rng = np.random.default_rng(14)
    dY = (rng.standard_normal((24, 128)) * np.exp(rng.normal(0, 2, (24, 1)))).astype(np.float32)   # [tokens, d_out]
    W = (rng.standard_normal((128, 96)) * 0.02).astype(np.float32)                                  # [d_out, d_in]
    cg, sg = oracle.quantize(dY, fg)            # blocks along d_out (the contraction)
    cw, sw = oracle.quantize(W, fw)             # forward codes: blocks along d_in
    Bc = np.ascontiguousarray(cw.T)             # B = W^T [d_in, d_out] for dX = dY W
    Bs = oracle.expand_scales(sw, axis=0)       # [d_in, d_out]: scale of the block along d_in
    C = oracle.gemm_exact_mixed(cg, oracle.expand_scales(sg), fg, Bc, Bs, fw)
    dg = _deq_exact64(cg, sg, fg)
    dw = _deq_exact64(cw, sw, fw)               # [d_out, d_in], reconstructed in its own layout
    ref = dg @ dw
    absmm = np.abs(dg) @ np.abs(dw)
    assert C.shape == (24, 96)
    assert np.all(np.abs(C - ref) <= 1e-13 * absmm)


RADIX_MIXED = [("E5C2", "E4C3_r8/9"), ("E4C3_r3/4", "E4C3_r8/9"), ("E4C3_r8/9", "E4C3"), ("E4C3_r3/4", "E3C3")]


@pytest.mark.parametrize("pair", RADIX_MIXED, ids=lambda p: f"{p[0]}x{p[1]}")
def test_mixed_rational_closure_all_pairs(pair):
    """Two lattices 2^(p_x n / N_x) and 2^(p_w n / N_w): every pair of nonzero codes, both
    signs, two scale pairs.  The product exponent, added as exact rationals, must equal
    t + h / H of the address on the common lattice; every one of its H phases is occupied, and
    H = lcm(N_x, N_w) / gcd of the lifted multipliers (8 for two binary radices, 36 for 2^(8/9)
    with E5C2's 2^(1/4), 72 with 2^(3/32))."""
    fx, fw = oracle.get_format(pair[0]), oracle.get_format(pair[1])
    D, lx, lw, g, H = oracle.mixed_lattice(fx, fw)

    def codes_of(f):
        mags = np.arange(1, 2 ** (f.E + f.C))
        return np.concatenate([mags, mags | (1 << (f.E + f.C))])

    cx, cw = codes_of(fx), codes_of(fw)
    _, sx, nx = oracle.code_fields(cx, fx)
    _, sw, nw = oracle.code_fields(cw, fw)
    phases = set()
    for ax, aw in [(0, 0), (-7, 4)]:
        for i in range(len(cx)):
            for j in range(len(cw)):
                d, h, t = oracle.product_address_mixed(int(cx[i]), ax, fx, int(cw[j]), aw, fw)
                q = Fraction(ax + aw) + Fraction(fx.p * int(nx[i]), fx.N) + Fraction(fw.p * int(nw[j]), fw.N)
                assert Fraction(t) + Fraction(h, H) == q
                assert 0 <= h < H and d == (-1 if sx[i] ^ sw[j] else 1)
                phases.add(h)
    assert phases == set(range(H))
    expect_H = {("E5C2", "E4C3_r8/9"): 36, ("E4C3_r3/4", "E4C3_r8/9"): 288, ("E4C3_r8/9", "E4C3"): 72,
                ("E4C3_r3/4", "E3C3"): 32}[pair]
    assert H == expect_H


@pytest.mark.parametrize("pair", RADIX_MIXED, ids=lambda p: f"{p[0]}x{p[1]}")
def test_mixed_rational_gemm_matches_float64_matmul(pair):
    fa, fb = oracle.get_format(pair[0]), oracle.get_format(pair[1])
    rng = np.random.default_rng(15)
    A = (rng.standard_normal((24, 160)) * np.exp(rng.normal(0, 3, (24, 1)))).astype(np.float32)
    B = (rng.standard_normal((20, 160)) * 0.02).astype(np.float32)
    ca, sa = oracle.quantize(A, fa)
    cb, sb = oracle.quantize(B, fb)
    C = oracle.gemm_exact_mixed(ca, oracle.expand_scales(sa), fa, cb, oracle.expand_scales(sb), fb)
    da, db = _deq_exact64(ca, sa, fa), _deq_exact64(cb, sb, fb)
    absmm = np.abs(da) @ np.abs(db).T
    assert np.all(np.abs(C - da @ db.T) <= 1e-13 * absmm)


# ------------------------------------------------------------------ static-operand MSE scales (Sec. 3.1)

def _exact_block_error(block, a, f):
    """Exact squared reconstruction error of one block at scale a (Fractions), with the codes from
    the rigorous nearest-level rule and the fp32 reconstruction rounded rigorously."""
    tot = Fraction(0)
    for v in block:
        v = float(v)
        if v == 0.0:
            continue
        y = abs(v) * 2.0 ** (-a)                       # exact: a power-of-two rescale of an fp32
        m, e = math.frexp(y)                            # y = m 2^e, m in [0.5, 1)
        M, j = int(m * (1 << 24)), e - 1
        n = X.nearest_level(M, j, f.E, f.C, f.p, f.q) if M >= (1 << 23) else None
        xh = 0.0 if n is None else math.copysign(X.rn_f32_level(a, n, f.p, f.N), v)
        if math.isinf(xh):
            return None                                 # the reconstruction overflows fp32
        tot += (Fraction(v) - Fraction(xh)) ** 2
    return tot


def _mse_blocks(seed):
    """Blocks where a lower scale can win: heavy tails, single outliers, a clipped top."""
    rng = np.random.default_rng(seed)
    b = [rng.standard_t(2, (24, 32)), rng.standard_normal((24, 32)),
         np.where(rng.random((24, 32)) < 0.05, 40.0, 1.0) * rng.standard_normal((24, 32))]
    return (np.concatenate(b) * 0.03).astype(np.float32)


@pytest.mark.parametrize("name", ALL_NAMES)
def test_mse_scale_is_the_exact_argmin(name):
    """The chosen scale minimizes the exact squared error over the candidates (a_c .. a_c - 3 and,
    when the level pattern spans P > 1 octaves, a_c + 1 .. a_c + P - 1), computed with exact
    Fractions of rigorously reconstructed values; a winner within 1e-12 of the best exact error
    is accepted (the float64 sum decides near-ties), and an exact tie keeps the first tried."""
    f = oracle.get_format(name)
    offs = oracle.mse_candidates(f, 4)
    assert offs[:4] == [0, -1, -2, -3] and len(offs) == 4 + (f.p // math.gcd(f.p, f.N)) - 1
    x = _mse_blocks(21)
    codes, scales = oracle.quantize_mse(x, f, candidates=4)
    _, s_ceil = oracle.quantize(x, f)
    moved = 0
    for r in range(x.shape[0]):
        ac = int(s_ceil[r, 0])
        errs = {}
        for u in offs:
            e = _exact_block_error(x[r], ac + u, f)
            if e is not None:
                errs[ac + u] = e
        best = min(errs.values())
        got = int(scales[r, 0])
        assert errs[got] <= best * (1 + Fraction(1, 10 ** 12)), (r, got, errs)
        first = next(ac + u for u in offs if ac + u in errs and errs[ac + u] == errs[got])
        assert got == first
        moved += got != ac
    # the search changes something on this data for the narrow formats
    if name in ("E3C3", "E4C3_r3/4"):
        assert moved > 0


@pytest.mark.parametrize("name", ALL_NAMES)
def test_mse_scales_beyond_the_candidates_never_better(name):
    """The reading behind the candidate set: a scale one whole level pattern above a candidate
    at or above a_c (a_c + P + j against a_c + j) never has a smaller exact error; and for binary
    radix and 2^(8/9) (P = 1) this rules out every scale above a_c."""
    f = oracle.get_format(name)
    P = f.p // math.gcd(f.p, f.N)
    x = _mse_blocks(22)[::3]
    _, s_ceil = oracle.quantize(x, f)
    for r in range(x.shape[0]):
        ac = int(s_ceil[r, 0])
        for j in range(P):
            e0, e1 = _exact_block_error(x[r], ac + j, f), _exact_block_error(x[r], ac + j + P, f)
            assert e0 is not None and e1 is not None and e1 >= e0, (r, j)


@pytest.mark.parametrize("name", ALL_NAMES)
def test_mse_special_cases(name):
    """One candidate is ceil-absmax; a block of representable values gets ceil-absmax's scale and
    codes (zero error, ties keep the first tried); zero and non-finite blocks as quantize()."""
    f = oracle.get_format(name)
    rng = np.random.default_rng(23)
    x = (rng.standard_normal((16, 256)) * np.exp2(rng.uniform(-20, 20, (16, 1)))).astype(np.float32)
    P = f.p // math.gcd(f.p, f.N)
    c1, s1 = oracle.quantize_mse(x, f, 1)
    c0, s0 = oracle.quantize(x, f)
    if P == 1:        # one candidate, and no scale above a_c to try: ceil-absmax itself
        assert np.array_equal(c1, c0) and np.array_equal(s1, s0)
    else:             # candidates counts the scales at or below a_c; a_c + 1 .. a_c + P - 1 remain
        d = s1.astype(int) - s0.astype(int)
        assert np.all((d >= 0) & (d < P))
    codes, scales = oracle.quantize(x, f)
    deq = oracle.dequantize(codes, scales, f)
    # reconstructed values are representable, so the search finds a zero-error scale and the
    # values come back exactly.  With P = 1 that scale is their own ceil-absmax scale (its
    # lattice contains the one they came from), and ties keep it; with 2^(3/4) halving the scale
    # moves the lattice, so ceil-absmax can lose them where the search does not
    c1, s1 = oracle.quantize(deq, f)
    c2, s2 = oracle.quantize_mse(deq, f, candidates=8)
    assert np.array_equal(oracle.dequantize(c2, s2, f), deq)
    if P == 1:
        assert np.array_equal(s2, s1) and np.array_equal(c2, c1)
    else:
        assert not np.array_equal(oracle.dequantize(c1, s1, f), deq)
    z = np.zeros((2, 64), np.float32)
    z[1, 3] = np.nan
    z[1, 40] = 1.0
    cz, sz = oracle.quantize_mse(z, f)
    assert list(sz[0]) == [-127, -127] and list(sz[1]) == [-128, sz[1, 1]] and np.all(cz[:, :32] == 0)
    a_c = int(oracle.quantize(z, f)[1][1, 1])
    assert sz[1, 1] == a_c if P == 1 else a_c <= sz[1, 1] < a_c + P


def test_mse_error_sum_order():
    """block_sq_error is the float64 sum in index order: it differs from a reordered sum on data
    built so the order matters, and matches a literal Python loop."""
    x = np.array([[2.0 ** 27] + [1.0] * 31], np.float64)   # 2^54 then 31 ones: in index order
    # each 1 is below half an ulp of the running sum and is lost; reversed, they add up first
    xh = np.zeros_like(x)
    e = oracle.block_sq_error(x, xh)[0]
    acc = 0.0
    for v in x[0]:
        acc = acc + v * v
    assert e == acc == 2.0 ** 54
    rev = 0.0
    for v in x[0][::-1]:
        rev = rev + v * v
    assert rev == 2.0 ** 54 + 32


@pytest.mark.parametrize("name", ["E4C3", "E5C2", "E3C3"])
def test_gemm_nonfinite_rows_are_nan(name):
    """A NaN or infinity in a block poisons it (scale -128, zero codes) and it reconstructs to
    NaN; the exact GEMM is deq(A) deq(B)^T in IEEE terms, so every output in a row of A or a
    column of B that holds a poisoned block is NaN (0 * NaN is NaN), and the other outputs are
    the products of the finite rows, as a float64 matmul of the reconstructed values gives."""
    f = oracle.get_format(name)
    rng = np.random.default_rng(17)
    A = rng.standard_normal((12, 96)).astype(np.float32)
    B = rng.standard_normal((10, 96)).astype(np.float32)
    A[3, 5] = np.nan
    A[7, 70] = np.inf
    B[2, 40] = -np.inf
    B[:, :32] = 0.0                       # B zero under A's poisoned block of row 3
    ca, sa = oracle.quantize(A, f)
    cb, sb = oracle.quantize(B, f)
    V = oracle.gemm_exact(ca, sa, cb, sb, f)
    da, db = oracle.dequantize(ca, sa, f), oracle.dequantize(cb, sb, f)
    nan_rows, nan_cols = np.isnan(da).any(1), np.isnan(db).any(1)
    assert list(np.nonzero(nan_rows)[0]) == [3, 7] and list(np.nonzero(nan_cols)[0]) == [2]
    assert np.array_equal(np.isnan(V), nan_rows[:, None] | nan_cols[None, :])
    keep_r, keep_c = ~nan_rows, ~nan_cols
    ref = _deq_exact64(ca[keep_r], sa[keep_r], f) @ _deq_exact64(cb[keep_c], sb[keep_c], f).T
    assert np.allclose(V[keep_r][:, keep_c], ref, rtol=1e-13, atol=0)
    # the tiny pure-Python oracle follows the same rule
    Vp = oracle.gemm_exact_python(ca[:5], sa[:5], cb[:4], sb[:4], f)
    assert np.array_equal(np.isnan(Vp), np.isnan(V[:5, :4]))
