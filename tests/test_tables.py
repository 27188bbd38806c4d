"""Host checks of the library's compile-time constant tables.

The build runs a table generator (csrc/gen_tables.cpp over the derivation in
csrc/tables.cpp, x87 exp2l with margin checks) and compiles its output into the
kernels.  These tests build the generator on its own, read its report and pin
what the tables encode against values derived here in 60-digit arithmetic
(mpmath), independently of the generator, and against the values the level
definition fixes (Sec. 3.1, Eq. curvefp-value: levels 2^{n/K}, K = 2^C; the
nearest-level rule's decision points are the midpoints between consecutive
levels and half the smallest level):

* every decision point (octave, 24-bit significand threshold) of every format;
* the fl32 mantissas of the levels 2^{f/N} (the dequantizer's and the
  ceil-absmax comparison's), for the binary and the rational radices;
* the GEMM expansion pairs hi = RN16(v), lo = RN16(v - hi) of every code byte.

The binary formats' thresholds are also compared with literal values
(significand thresholds of the midpoints (2^{h/K} + 2^{(h+1)/K}) / 2 for
K = 8 and 4, and of the zero points 2^{n_min/K - 1}) that were worked out by
hand from the same definition.
"""

import os
import subprocess
import tempfile

import mpmath
import pytest

from paper_2608_10010_amd import build as B

mpmath.mp.dps = 60

# (E, C, p, q) per format id of the C ABI
FORMATS = {0: (4, 3, 1, 1), 1: (5, 2, 1, 1), 2: (3, 3, 1, 1), 3: (4, 3, 8, 9), 4: (4, 3, 3, 4)}

# significand thresholds in [2^23, 2^24) of the midpoints between 2^{h/K} and 2^{(h+1)/K}
T_K8 = [8768224, 9561817, 10427235, 11370980, 12400142, 13522451, 14746337, 16080995]
T_K4 = [9182200, 10919537, 12985591, 15442558]
# zero points 2^{n_min/K - 1}: (octave, threshold)
ZERO = {0: (-9, 9147841), 1: (-17, 9975792), 2: (-5, 9147841)}
# fp32 bits of fl32(2^{k/8}) and fl32(2^{k/4})
FL32_K8 = [0x3F800000, 0x3F8B95C2, 0x3F9837F0, 0x3FA5FED7, 0x3FB504F3, 0x3FC5672A, 0x3FD744FD, 0x3FEAC0C7]
FL32_K4 = [0x3F800000, 0x3F9837F0, 0x3FB504F3, 0x3FD744FD]


@pytest.fixture(scope="module")
def report():
    with tempfile.TemporaryDirectory() as d:
        exe = B.build_generator(d)
        out = subprocess.run([exe, "--report"], capture_output=True, text=True, check=True).stdout
        # the generator also writes the include file the kernels are compiled with
        inc = os.path.join(d, "t.inc")
        subprocess.run([exe, inc], check=True)
        inc_text = open(inc).read()
    rep, cur = {}, None
    for line in out.splitlines():
        f = line.split()
        if f[0] == "format":
            cur = int(f[1])
            rep[cur] = {"mid": {}, "dq_em": {}, "dec": {}, "hdr": dict(kv.split("=") for kv in f[3:])}
        elif f[0] == "zero":
            rep[cur]["zero"] = (int(f[1]), int(f[2]), int(f[3]))
        elif f[0] == "mid":
            rep[cur]["mid"][int(f[1])] = (int(f[2]), int(f[3]))
        else:
            rep[cur][f[0]][int(f[1])] = int(f[2], 16)
    return rep, inc_text


def params(fid):
    E, C, p, q = FORMATS[fid]
    K = 1 << C
    B_ = 1 << (E + C - 1)
    return E, C, p, q, K, q * K, -(B_ - 1), B_ - 1, B_


def level(fid, n):
    _, _, p, _, _, N, _, _, _ = params(fid)
    return mpmath.power(2, mpmath.mpf(p * n) / N)


def point(v):
    """(octave, floor of the 24-bit significand) of a positive irrational v."""
    o = int(mpmath.floor(mpmath.log(v, 2)))
    return o, int(mpmath.floor(mpmath.ldexp(v, 23 - o)))


def rn_bits32(v):
    """fp32 bits of the nearest float (normal range, v > 0, never a tie)."""
    o = int(mpmath.floor(mpmath.log(v, 2)))
    m = int(mpmath.nint(mpmath.ldexp(v, 23 - o)))
    if m == 1 << 24:
        m, o = 1 << 23, o + 1
    return ((o + 127) << 23) | (m - (1 << 23))


def rn16(v):
    """(fp16 bits, value) of the nearest fp16 of v >= 0 (ties to even; subnormals included)."""
    if v == 0:
        return 0, mpmath.mpf(0)
    o = int(mpmath.floor(mpmath.log(v, 2)))
    sh = 10 - o if o >= -14 else 24
    x = mpmath.ldexp(v, sh)
    fl = int(mpmath.floor(x))
    fr = x - fl
    m = fl + (1 if fr > 0.5 or (fr == 0.5 and fl & 1) else 0)
    val = mpmath.ldexp(m, -sh)
    if o >= -14:
        if m == 2048:
            m, o = 1024, o + 1
        return ((o + 15) << 10) | (m - 1024), val
    return m, val


@pytest.mark.parametrize("fid", [0, 1, 2])
def test_binary_thresholds_match_hand_values(report, fid):
    rep, _ = report
    _, _, _, _, K, _, nmin, nmax, _ = params(fid)
    T = T_K8 if K == 8 else T_K4
    mids = rep[fid]["mid"]
    assert len(mids) == nmax - nmin
    for i, (o, t) in mids.items():
        n = nmin + i                       # between n and n + 1
        h = n % K
        assert t == T[h], (fid, i)
        assert o == n // K, (fid, i)
    assert rep[fid]["zero"] == ZERO[fid] + (0,)


@pytest.mark.parametrize("fid", sorted(FORMATS))
def test_every_decision_point(report, fid):
    rep, _ = report
    _, _, _, _, _, N, nmin, nmax, _ = params(fid)
    mids = rep[fid]["mid"]
    assert sorted(mids) == list(range(nmax - nmin))
    for i in range(nmax - nmin):
        n = nmin + i
        assert mids[i] == point((level(fid, n) + level(fid, n + 1)) / 2), (fid, n)
    zo, zt, zexact = rep[fid]["zero"]
    half = level(fid, nmin) / 2
    _, _, p, _, _, N, _, _, _ = params(fid)
    if (p * nmin) % N == 0:
        # the smallest level is a power of two (r = 2^(8/9): 2^-7): its half is a float
        assert zexact == 1 and (zo, zt) == (int(mpmath.log(half, 2)), 1 << 23)
    else:
        assert zexact == 0 and (zo, zt) == point(half)


@pytest.mark.parametrize("fid", sorted(FORMATS))
def test_level_mantissas(report, fid):
    rep, _ = report
    _, _, p, _, K, N, nmin, nmax, B_ = params(fid)
    em = rep[fid]["dq_em"]
    for m in range(1, 2 * B_):
        u = p * (m - B_)
        w, f = u // N, u % N
        bits = rn_bits32(mpmath.power(2, mpmath.mpf(f) / N))
        assert em[m] & 0x7FFFFF == bits & 0x7FFFFF, (fid, m)
        assert (em[m] >> 24) == (w & 0xFF), (fid, m)
        assert (bits >> 23) in (127, 128)
    # fl32 of the top level: the ceil-absmax comparison value
    top = rn_bits32(level(fid, nmax))
    assert int(rep[fid]["hdr"]["lmax_mant"], 16) == top & 0x7FFFFF
    if p == 1:
        fl = FL32_K8 if K == 8 else FL32_K4
        for k in range(K):
            m = B_ + k                     # n = k
            assert (0x3F800000 | em[m] & 0x7FFFFF) == fl[k]


@pytest.mark.parametrize("fid", sorted(FORMATS))
def test_expansion_pairs(report, fid):
    rep, _ = report
    E, C, p, q, K, N, nmin, nmax, B_ = params(fid)
    ohi = (p * nmax) // N
    bias = 15 - ohi
    dec = rep[fid]["dec"]
    for code in range(256):
        m = code & (2 * B_ - 1)
        s = (code >> (E + C)) & 1
        if code >= (1 << (E + C + 1)):
            continue                       # not a code of this width
        if m == 0:
            assert dec[code] == 0          # both zero codes expand to (+0, +0)
            continue
        u = p * (m - B_)
        w, f = u // N, u % N
        v = mpmath.ldexp(mpmath.power(2, mpmath.mpf(f) / N), w + bias)
        hb, hv = rn16(v)
        rest = v - hv
        lb, _ = rn16(abs(rest))
        if lb and rest < 0:
            lb |= 0x8000
        if s:
            hb ^= 0x8000
            if lb:
                lb ^= 0x8000
        assert dec[code] == (lb << 16) | hb, (fid, code)


def test_include_file_holds_the_reported_tables(report):
    """The include file the kernels compile is written from the same derivation: spot-check that
    every binary format's level mantissas and expansion pairs appear in it."""
    rep, inc = report
    assert "CURVEFP_QLUT_INIT" in inc and "CURVEFP_DEC_INIT" in inc
    for fid in (0, 1, 2):
        assert f"0x{rep[fid]['dec'][0x40 | 1]:08x}u" in inc
        assert f"0x{int(rep[fid]['hdr']['lmax_mant'], 16):06x}u" in inc
