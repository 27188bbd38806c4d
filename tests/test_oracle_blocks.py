"""Oracle pins for block sizes G other than 32 (Eq. effective-rate's G; Sec. 3.1 evaluates
fixed-size blocks and rowwise sharing, Sec. 4.2 uses G64 and G512).

Each block of G consecutive elements gets one ceil-absmax scale and every element the nearest
level at that scale.  These tests hold the oracle to that definition through facts that do
not come from its own code:
  * the scale rule is monotone in the block maximum, so a block's scale is the largest of the
    scales its groups of 32 get alone (an all-zero group takes the bottom of the range, -127:
    every integer satisfies the ceil-absmax inequality for a zero maximum);
  * every code is the nearest level at the block scale, decided by the rigorous integer
    brackets of tests/exact_ref.py;
  * the exact GEMM over blocks of G equals numpy's float64 product of the dequantized operands
    within fp64 rounding, and equals the exact GEMM at G = 32 with each scale repeated.
"""

import math

import numpy as np
import pytest

import oracle
from tests import exact_ref

NAMES = list(oracle.FORMATS)
BLOCKS = [64, 128, 256, 512, 96, 160]


def sample_input(rng, rows, cols):
    """Groups of 32 with magnitudes spread over 2^-20 .. 2^20, some groups all zero."""
    x = rng.standard_normal((rows, cols)) * np.exp2(rng.uniform(-20, 20, (rows, cols // 32, 1))).repeat(32, 1).reshape(
        rows, cols // 32, 32).reshape(rows, cols)
    zero = rng.random((rows, cols // 32)) < 0.15
    x = np.where(np.repeat(zero, 32, axis=1), 0.0, x)
    return x.astype(np.float32)


def rigorous_code(x: float, a: int, f) -> int:
    """Code of the nearest element of {0} U {2^(a + p n / (qK))} to x (exact_ref brackets)."""
    if x == 0:
        return 0
    m, e = math.frexp(abs(x))            # |x| = m 2^e, m in [0.5, 1)
    M = int(m * (1 << 24))               # exact: fp32 has 24 significand bits
    n = exact_ref.nearest_level(M, e - 1 - a, f.E, f.C, f.p, f.q)
    if n is None:
        return 0
    return ((1 if x < 0 else 0) << (f.E + f.C)) | (n + f.B)


@pytest.mark.parametrize("name", NAMES)
@pytest.mark.parametrize("G", BLOCKS + ["row"])
def test_block_scale_is_largest_group_scale(name, G):
    f = oracle.get_format(name)
    rng = np.random.default_rng(40 + len(name))
    cols = 960
    G = cols if G == "row" else G
    if cols % G:
        cols = 2 * G * 3
    x = sample_input(rng, 12, cols)
    _, sg = oracle.quantize(x, f, G)
    _, s32 = oracle.quantize(x, f, 32)
    groups = np.abs(x).reshape(12, cols // 32, 32).max(-1) > 0
    assert (~groups).any() and np.all(s32[~groups] == -127)
    expect = s32.astype(np.int64).reshape(12, cols // G, G // 32).max(-1)
    assert sg.shape == (12, cols // G)
    assert np.array_equal(sg.astype(np.int64), expect)


@pytest.mark.parametrize("name", NAMES)
@pytest.mark.parametrize("G", [64, 512, 96])
def test_block_codes_are_nearest_at_block_scale(name, G):
    f = oracle.get_format(name)
    rng = np.random.default_rng(7 + G)
    cols = 2 * G * 3 if G == 96 else 2 * G
    x = sample_input(rng, 4, cols)
    codes, scales = oracle.quantize(x, f, G)
    a = np.repeat(scales.astype(np.int64), G, axis=1)
    idx = rng.choice(x.size, 400, replace=False)
    for i in idx:
        r, c = divmod(int(i), cols)
        assert int(codes[r, c]) == rigorous_code(float(x[r, c]), int(a[r, c]), f), (r, c, float(x[r, c]))


@pytest.mark.parametrize("name", NAMES)
def test_block_round_trip(name):
    """Quantizing the reconstruction of blocks of G: the largest element's level lies in the top
    octave of the block's range or one octave lower, so the scale stays or drops by one (it can
    drop when that level is a whole octave below the top: its value is at most
    2^(a-1) fl32(L_max)); blocks that keep their scale give back their codes."""
    f = oracle.get_format(name)
    rng = np.random.default_rng(3)
    for G in (64, 256, 512):
        x = sample_input(rng, 6, 1024)
        c, s = oracle.quantize(x, f, G)
        xh = oracle.dequantize(c, s, f, G)
        c2, s2 = oracle.quantize(xh, f, G)
        d = s.astype(np.int64) - s2.astype(np.int64)
        assert set(np.unique(d)) <= {0, 1}, G
        keep = np.repeat(d == 0, G, axis=1)
        assert np.array_equal(np.where(keep, c, 0), np.where(keep, c2, 0)), G
        assert (d == 0).mean() > 0.5, G


def test_block_nonfinite_poisons_the_whole_block():
    f = oracle.get_format("E4C3")
    x = np.ones((2, 256), np.float32)
    x[0, 200] = np.inf
    codes, scales = oracle.quantize(x, f, 128)
    assert scales[0, 1] == oracle.POISON_SCALE and not codes[0, 128:].any()
    assert scales[0, 0] != oracle.POISON_SCALE and scales[1].tolist() == [scales[0, 0]] * 2


@pytest.mark.parametrize("name", NAMES)
@pytest.mark.parametrize("G", [64, 256, 96])
def test_gemm_over_blocks_of_g(name, G):
    f = oracle.get_format(name)
    rng = np.random.default_rng(50 + G)
    K = 3 * G if G == 96 else 2 * G
    A = sample_input(rng, 9, K)
    B = sample_input(rng, 7, K)
    ca, sa = oracle.quantize(A, f, G)
    cb, sb = oracle.quantize(B, f, G)
    V = oracle.gemm_exact(ca, sa, cb, sb, f, block=G)
    # the same products at G = 32 with each block scale repeated: the exact sums agree exactly
    r = G // 32
    V32 = oracle.gemm_exact(ca, np.repeat(sa, r, axis=1), cb, np.repeat(sb, r, axis=1), f, block=32)
    assert np.array_equal(V, V32)
    # and numpy's float64 product of the reconstructions, within fp64 rounding
    da = oracle.dequantize(ca, sa, f, G).astype(np.float64)
    db = oracle.dequantize(cb, sb, f, G).astype(np.float64)
    # fp32 reconstruction differs from the exact level by at most 2^-24 relative per operand
    ref = da @ db.T
    bound = (2.0 ** -22 + K * 2.0 ** -52) * (np.abs(da) @ np.abs(db).T) + 2.0 ** -140
    assert np.all(np.abs(V - ref) <= bound)


@pytest.mark.parametrize("pair", [("E5C2", "E4C3"), ("E4C3_r3/4", "E4C3_r8/9")], ids=lambda p: f"{p[0]}x{p[1]}")
def test_mixed_gemm_with_reused_operand_in_blocks_of_g(pair):
    """The backward recipe with blocks of 64: A quantized along K, B a reused [K][N] operand whose
    blocks of 64 run along N; per-element scales expand both."""
    fa, fb = (oracle.get_format(n) for n in pair)
    rng = np.random.default_rng(61)
    G, M, N, K = 64, 5, 128, 128
    A = sample_input(rng, M, K)
    Bt = sample_input(rng, K, N)                  # [K][N], quantized along N
    ca, sa = oracle.quantize(A, fa, G)
    cbt, sbt = oracle.quantize(Bt, fb, G)
    ea = oracle.expand_scales(sa, G, axis=1)
    eb = oracle.expand_scales(sbt, G, axis=0)     # [N][K]
    cb = np.ascontiguousarray(cbt.T)
    V = oracle.gemm_exact_mixed(ca, ea, fa, cb, eb, fb)
    da = oracle.dequantize(ca, sa, fa, G).astype(np.float64)
    db = oracle.dequantize(cbt, sbt, fb, G).astype(np.float64).T
    ref = da @ db.T
    bound = (2.0 ** -22 + K * 2.0 ** -52) * (np.abs(da) @ np.abs(db).T) + 2.0 ** -140
    assert np.all(np.abs(V - ref) <= bound)


# ---------------------------------------------------------------- S-bit scale exponents

def spread_rows(rng, rows, cols, G, spread):
    """Blocks of G along rows with block magnitudes 2^U(0, spread) below a row top of 2^U(-5, 5)."""
    top = rng.uniform(-5, 5, (rows, 1))
    blk = top - rng.uniform(0, spread, (rows, cols // G))
    x = rng.standard_normal((rows, cols)) * np.exp2(np.repeat(blk, G, axis=1))
    return x.astype(np.float32)


@pytest.mark.parametrize("name", NAMES)
@pytest.mark.parametrize("S", [4, 5])
def test_compact_within_window_is_the_block_quantizer(name, S):
    """When every block's scale lies within 2^S - 2 of its row's largest, the S-bit form holds the
    block quantizer's codes and scales exactly (reference - offset)."""
    f = oracle.get_format(name)
    rng = np.random.default_rng(70 + S)
    G = 64
    x = spread_rows(rng, 8, 1024, G, (1 << S) - 6)
    c, s = oracle.quantize(x, f, G)
    cc, ref, d = oracle.quantize_compact(x, f, G, S)
    assert np.array_equal(cc, c)
    assert np.array_equal(oracle.compact_scales(ref, d, S), s)
    assert ref.tolist() == s.astype(np.int64).max(axis=1).tolist()
    assert d.max() <= (1 << S) - 2


@pytest.mark.parametrize("name", NAMES)
def test_compact_raised_blocks_are_nearest_at_the_raised_scale(name):
    f = oracle.get_format(name)
    rng = np.random.default_rng(77)
    G, S = 64, 4
    x = spread_rows(rng, 4, 512, G, 40)          # blocks far below the row top
    cc, ref, d = oracle.quantize_compact(x, f, G, S)
    _, s = oracle.quantize(x, f, G)
    window = (1 << S) - 2
    raised = s.astype(np.int64) < ref.astype(np.int64)[:, None] - window
    assert raised.any() and np.all(d[raised] == window)
    a = np.repeat(oracle.compact_scales(ref, d, S).astype(np.int64), G, axis=1)
    for r, c in zip(*np.nonzero(np.repeat(raised, G, axis=1))):
        if rng.random() < 0.25:
            assert int(cc[r, c]) == rigorous_code(float(x[r, c]), int(a[r, c]), f), (r, c)


def test_compact_markers_zero_blocks_and_rows():
    f = oracle.get_format("E3C3")
    x = np.ones((3, 256), np.float32) * np.float32(3.0)
    x[0, 70] = np.nan                     # block 1 of row 0 poisoned
    x[1, :64] = 0.0                       # block 0 of row 1 all zero
    x[2, :] = 0.0                         # an all-zero row
    x[1, 64:] = np.float32(2.0 ** -30)    # row 1's other blocks far below nothing: they set the reference
    for S in (4, 5):
        cc, ref, d = oracle.quantize_compact(x, f, 64, S)
        _, s = oracle.quantize(x, f, 64)
        assert d[0].tolist() == [0, (1 << S) - 1, 0, 0] and not cc[0, 64:128].any()
        assert ref[0] == s[0, 0]
        assert d[1, 0] == 0 and ref[1] == s[1, 1] and not cc[1, :64].any()
        assert ref[2] == 0 and d[2].tolist() == [0, 0, 0, 0] and not cc[2].any()
        assert oracle.compact_scales(ref, d, S)[0, 1] == oracle.POISON_SCALE


def test_compact_offset_packing_layout():
    """Offsets LSB first in a little-endian bit string, rows padded to whole bytes, worked by
    hand: S = 4, offsets 1, 2, 15, 0, 7 -> 0x21 0x0F 0x07; S = 5, offsets 1, 2, 31, 4 -> bits 0
    (1), 6 (2 << 5), 10..14 (31 << 10), 17 (4 << 15) -> 0x41 0x7C 0x02."""
    assert oracle.pack_offsets(np.array([[1, 2, 15, 0, 7]]), 4).tolist() == [[0x21, 0x0F, 0x07]]
    assert oracle.pack_offsets(np.array([[1, 2, 31, 4]]), 5).tolist() == [[0x41, 0x7C, 0x02]]
    rng = np.random.default_rng(5)
    for S in range(2, 9):
        d = rng.integers(0, 1 << S, (3, 37))
        p = oracle.pack_offsets(d, S)
        assert p.shape == (3, (37 * S + 7) // 8)
        assert np.array_equal(oracle.unpack_offsets(p, 37, S), d)


# ---------------------------------------------------------------- tensorwise scales

@pytest.mark.parametrize("name", NAMES)
def test_tensorwise_scale_is_largest_row_scale(name):
    f = oracle.get_format(name)
    rng = np.random.default_rng(80)
    x = sample_input(rng, 9, 256)
    x[3] = 0.0                                    # an all-zero row takes no part
    c, s = oracle.quantize_tensorwise(x, f)
    _, sr = oracle.quantize(x, f, 256)
    live = np.abs(x).max(axis=1) > 0
    assert s.shape == (9, 1) and np.all(s == s[0, 0])
    assert int(s[0, 0]) == int(sr[live, 0].astype(np.int64).max())


@pytest.mark.parametrize("name", NAMES)
def test_tensorwise_codes_are_nearest_at_the_tensor_scale(name):
    f = oracle.get_format(name)
    rng = np.random.default_rng(81)
    x = sample_input(rng, 5, 512)
    c, s = oracle.quantize_tensorwise(x, f)
    a = int(s[0, 0])
    for i in rng.choice(x.size, 300, replace=False):
        r, k = divmod(int(i), 512)
        assert int(c[r, k]) == rigorous_code(float(x[r, k]), a, f), (r, k)


@pytest.mark.parametrize("name", NAMES)
def test_tensorwise_equals_rowwise_when_rows_share_their_maximum(name):
    """Rows scaled to the same largest magnitude: the tensor's scale is every row's."""
    f = oracle.get_format(name)
    rng = np.random.default_rng(82)
    x = rng.standard_normal((6, 128)).astype(np.float64)
    x = x / np.abs(x).max(axis=1, keepdims=True) * 3.5
    x = x.astype(np.float32)
    c, s = oracle.quantize_tensorwise(x, f)
    cr, sr = oracle.quantize(x, f, 128)
    assert np.array_equal(c, cr) and np.array_equal(s, sr)


def test_tensorwise_nonfinite_poisons_the_tensor():
    f = oracle.get_format("E4C3")
    x = np.ones((4, 64), np.float32)
    x[2, 5] = np.inf
    c, s = oracle.quantize_tensorwise(x, f)
    assert np.all(s == oracle.POISON_SCALE) and not c.any()


# ---------------------------------------------------------------- static scales over blocks of G

@pytest.mark.parametrize("name", NAMES)
def test_mse_over_blocks_of_g_is_the_exact_argmin(name):
    """Static-operand scales with G = 64 (Sec. 4.2's PTQ weights): the chosen scale minimizes the
    exact squared error of the 64-element block over the candidates (exact Fractions of
    rigorously reconstructed values, as for blocks of 32); an exact tie keeps the first tried."""
    from fractions import Fraction
    from tests.test_oracle_pins import _exact_block_error, _mse_blocks
    f = oracle.get_format(name)
    x = np.ascontiguousarray(_mse_blocks(31).reshape(-1, 64)[::2])     # two 32-blocks per row
    offs = oracle.mse_candidates(f, 4)
    codes, scales = oracle.quantize_mse(x, f, candidates=4, block=64)
    _, s_ceil = oracle.quantize(x, f, 64)
    for r in range(x.shape[0]):
        ac = int(s_ceil[r, 0])
        errs = {ac + u: e for u in offs if (e := _exact_block_error(x[r], ac + u, f)) is not None}
        best = min(errs.values())
        got = int(scales[r, 0])
        assert errs[got] <= best * (1 + Fraction(1, 10 ** 12)), (r, got)
        assert got == next(ac + u for u in offs if ac + u in errs and errs[ac + u] == errs[got])
        # and the codes are the nearest levels at the chosen scale
        for i in range(0, 64, 7):
            assert int(codes[r, i]) == rigorous_code(float(x[r, i]), got, f), (r, i)
