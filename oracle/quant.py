"""Block quantizer Q(X) and reconstruction for CurveFP (oracle; test infrastructure only).

Plain numpy in float64.  Each function follows the paper's definition directly:

* reconstruction  x_hat = (-1)^s 2^{a_b} r^{e+k/K}             (Eq. curvefp-value)
* quantization    keep the sign, take the magnitude nearest to |x| in absolute
                  error, saturate at the endpoints                 (Sec. 3.1)
* block scale     dynamic operands use ceil-absmax scaling         (Sec. 3.1, App. A.2)

Readings taken where the paper is silent:

* ceil-absmax: a_b is the smallest integer a with amax <= 2^a * fl32(L_max),
  L_max = r^{n_max/K} the largest positive level.  fl32(L_max) is the value the
  top code actually reconstructs to, so a block that holds its own top code
  keeps its scale (quantize(dequantize(c)) == c).  All-zero block: every integer
  satisfies the inequality, so a_b is the bottom of the stored range, -127.
  a_b is stored as int8, clamped to [-127, 127].
* non-finite inputs: a block holding NaN or +-Inf gets scale -128 and all-zero
  codes; it reconstructs to NaN.
* the zero sentinel is the only zero: every zero result is code 0x00 (the
  source sign of a zero result is not kept).
* the candidate set for the nearest search is {0} U {levels}: a tiny value goes
  to zero when it is nearer to zero than to the smallest level.
* reconstruction to fp32 is the fp32 value nearest to the real x_hat.
* E3C3 codes are packed 7 bits each, LSB first: code i of a 32-element block
  occupies bits [7i, 7i+7) of a 224-bit little-endian string (28 bytes).
"""

import numpy as np

from .formats import Format

POISON_SCALE = -128
SCALE_MIN = -127
SCALE_MAX = 127


_SIG_CACHE = {}


def _sig_table(fmt: Format) -> np.ndarray:
    """S[r] = 2^{r/N} for r in [0, N), N = qK: the fractional part of every level, each the
    float64 nearest to the real value (evaluated with mpmath at 40 digits, then rounded once;
    ``2.0 ** (r / N)`` would round r / N first whenever N is not a power of two)."""
    N = fmt.N
    if N not in _SIG_CACHE:
        import mpmath
        with mpmath.workdps(40):
            _SIG_CACHE[N] = np.array([float(mpmath.power(2, mpmath.mpf(r) / N)) for r in range(N)],
                                     dtype=np.float64)
    return _SIG_CACHE[N]


def level_value_f64(fmt: Format, n):
    """r^{n/K} = 2^{p n / (qK)} in float64 (Sec. 3.2: r^{e+k/K} = 2^{p(eK+k)/(qK)}).

    Written as ldexp(S[u mod N], floor(u / N)) with u = p*n, so levels one
    octave apart differ by exactly a factor of two in float64 as well.
    """
    n = np.asarray(n, dtype=np.int64)
    u = fmt.p * n
    N = fmt.N
    frac = np.mod(u, N)
    whole = np.floor_divide(u, N)
    return np.ldexp(_sig_table(fmt)[frac], whole.astype(np.int64))


def top_level_fp32(fmt: Format) -> float:
    """fl32(L_max): the fp32 value of the largest level at scale 0."""
    return float(np.float32(level_value_f64(fmt, fmt.n_max)))


def scale_exponents(amax: np.ndarray, fmt: Format) -> np.ndarray:
    """Ceil-absmax block scale: smallest integer a with amax <= 2^a * fl32(L_max).

    ``amax`` holds the block maxima of |x| in float64 (exact copies of fp32
    values).  Zero blocks get SCALE_MIN (every a satisfies 0 <= 2^a fl32(L_max); the
    smallest stored one), non-finite blocks get POISON_SCALE, the rest is clamped to
    [-127, 127].  Returns int64.
    """
    amax = np.asarray(amax, dtype=np.float64)
    lm = top_level_fp32(fmt)
    finite = np.isfinite(amax)
    pos = finite & (amax > 0)
    safe = np.where(pos, amax, 1.0)
    a = np.ceil(np.log2(safe) - np.log2(lm)).astype(np.int64)
    # make a exact with two-sided checks (ldexp by an integer is exact in fp64)
    for _ in range(3):
        a = np.where(safe > np.ldexp(lm, a), a + 1, a)
        a = np.where(safe <= np.ldexp(lm, a - 1), a - 1, a)
    assert np.all(safe[pos] <= np.ldexp(lm, a[pos]))
    assert np.all(safe[pos] > np.ldexp(lm, a[pos] - 1))
    a = np.where(pos, a, SCALE_MIN)
    a = np.clip(a, SCALE_MIN, SCALE_MAX)
    a = np.where(finite, a, POISON_SCALE)
    return a.astype(np.int64)


def _nearest_index(y: np.ndarray, fmt: Format):
    """Nearest element of {0} U {r^{n/K}: n_min <= n <= n_max} to y >= 0.

    Returns (is_zero, n).  Candidates: zero, and the four levels around the
    continuous index floor(log_r(y) * K); the nearest is found by comparing
    absolute errors |y - level| (Sec. 3.1).  Values above the top level end up
    on n_max and values below the smallest level on n_min or zero, which is the
    saturation the paper asks for.
    """
    y = np.asarray(y, dtype=np.float64)
    with np.errstate(divide="ignore", invalid="ignore"):
        cont = np.floor(np.log2(np.where(y > 0, y, 1.0)) * fmt.N / fmt.p)
    cont = np.where(y > 0, cont, fmt.n_min).astype(np.int64)
    best_n = np.full(y.shape, fmt.n_min, dtype=np.int64)
    best_d = np.full(y.shape, np.inf)
    for d in (-1, 0, 1, 2):
        cand = np.clip(cont + d, fmt.n_min, fmt.n_max)
        dist = np.abs(y - level_value_f64(fmt, cand))
        take = dist < best_d
        best_n = np.where(take, cand, best_n)
        best_d = np.where(take, dist, best_d)
    is_zero = y < best_d  # |y - 0| < |y - nearest level|
    return is_zero, best_n


def quantize(x: np.ndarray, fmt: Format, block: int = 32):
    """Q(X) along the last axis in blocks of ``block`` consecutive elements.

    x: float32 array [outer, k] (bf16 sources are passed widened to fp32).
    Returns (codes uint8 [outer, k], scales int8 [outer, k // block]); codes
    are unpacked, one per byte, for every format.
    """
    x = np.asarray(x)
    assert x.dtype == np.float32 and x.ndim == 2
    outer, k = x.shape
    assert k % block == 0
    xb = x.astype(np.float64).reshape(outer, k // block, block)
    mag = np.abs(xb)
    with np.errstate(invalid="ignore"):
        finite_block = np.all(np.isfinite(xb), axis=-1)
    amax = np.where(finite_block, np.max(np.where(np.isfinite(mag), mag, 0.0), axis=-1), np.inf)
    a = scale_exponents(amax, fmt)
    a_safe = np.where(finite_block, a, 0)
    y = np.ldexp(np.where(np.isfinite(mag), mag, 0.0), -a_safe[..., None])
    is_zero, n = _nearest_index(y, fmt)
    sign = np.signbit(xb).astype(np.int64)
    m = n + fmt.B
    codes = (sign << (fmt.E + fmt.C)) | m
    codes = np.where(is_zero, 0, codes)
    codes = np.where(finite_block[..., None], codes, 0)
    return codes.reshape(outer, k).astype(np.uint8), a.astype(np.int8)


def _codes_at_scale(xb: np.ndarray, a: np.ndarray, fmt: Format) -> np.ndarray:
    """Codes of finite blocks xb [..., block] (float64 copies of the source) at the block
    scales a [...]: sign kept, magnitude nearest to |x| 2^-a, saturating (Sec. 3.1)."""
    y = np.ldexp(np.abs(xb), -a[..., None])
    is_zero, n = _nearest_index(y, fmt)
    codes = (np.signbit(xb).astype(np.int64) << (fmt.E + fmt.C)) | (n + fmt.B)
    return np.where(is_zero, 0, codes)


def _reconstruct_f32(codes: np.ndarray, a: np.ndarray, fmt: Format) -> np.ndarray:
    """fp32 reconstruction of block codes [..., block] at the block scales a [...]."""
    nz, s, n = code_fields(codes, fmt)
    mag = np.ldexp(level_value_f64(fmt, np.where(nz, n, 0)), a[..., None])
    val = np.where(nz, np.where(s == 1, -mag, mag), 0.0)
    with np.errstate(over="ignore"):
        return val.astype(np.float32)


def block_sq_error(xb: np.ndarray, xh: np.ndarray) -> np.ndarray:
    """Reconstruction error of each block: sum over i of (x_i - x_hat_i)^2, each step one
    float64 operation, i in index order (no fused multiply-add)."""
    d = xb.astype(np.float64) - xh.astype(np.float64)
    acc = np.zeros(d.shape[:-1], dtype=np.float64)
    with np.errstate(over="ignore", invalid="ignore"):
        for i in range(d.shape[-1]):
            acc = acc + d[..., i] * d[..., i]
    return acc


def mse_candidates(fmt: Format, candidates: int):
    """Scale offsets from the ceil-absmax scale a_c that the static search tries, in order:
    0, -1, ..., -(candidates - 1) (``candidates`` counts the scales at or below a_c), then
    +1, ..., +(P - 1), where P = p / gcd(p, qK) is the number
    of octaves after which the level pattern 2^(p n / (qK)) repeats (1 for binary radix and
    2^(8/9), 3 for 2^(3/4)).  A scale a_c + P + j is never better than a_c + j (j >= 0): its
    levels are those of a_c + j shifted up by a whole pattern, so it keeps every level up to the
    block's top and only drops levels at the bottom; within one pattern the lattices differ."""
    period = fmt.p // fmt.g
    return [-d for d in range(candidates)] + list(range(1, period))


def quantize_mse(x: np.ndarray, fmt: Format, candidates: int = 4, block: int = 32):
    """Q(X) with static-operand scales: each block takes the power-of-two scale among a_c + u,
    u in mse_candidates(fmt, candidates) (a_c the ceil-absmax scale; scales outside [-127, 127]
    are not tried), whose fp32 reconstruction has the least squared error (block_sq_error);
    a tie keeps the scale tried first (Sec. 3.1: a static operand's power-of-two scale is the one
    that minimizes the squared reconstruction error).  Zero blocks get scale -127, non-finite blocks -128, as in
    quantize().  Returns (codes, scales) like quantize()."""
    x = np.asarray(x)
    assert x.dtype == np.float32 and x.ndim == 2 and 1 <= candidates <= 8
    outer, k = x.shape
    assert k % block == 0
    xb = x.astype(np.float64).reshape(outer, k // block, block)
    mag = np.abs(xb)
    with np.errstate(invalid="ignore"):
        finite_block = np.all(np.isfinite(xb), axis=-1)
    amax = np.where(finite_block, np.max(np.where(np.isfinite(mag), mag, 0.0), axis=-1), np.inf)
    a_c = scale_exponents(amax, fmt)
    live = finite_block & (amax > 0)
    xs = np.where(finite_block[..., None], xb, 0.0)
    best_a = np.where(live, a_c, SCALE_MIN)
    best_codes = _codes_at_scale(xs, best_a, fmt)
    best_err = block_sq_error(xs, _reconstruct_f32(best_codes, best_a, fmt))
    for u in mse_candidates(fmt, candidates)[1:]:
        a = a_c + u
        ok = live & (a >= SCALE_MIN) & (a <= SCALE_MAX)
        a_try = np.where(ok, a, 0)
        codes = _codes_at_scale(xs, a_try, fmt)
        err = block_sq_error(xs, _reconstruct_f32(codes, a_try, fmt))
        take = ok & (err < best_err)
        best_a = np.where(take, a, best_a)
        best_codes = np.where(take[..., None], codes, best_codes)
        best_err = np.where(take, err, best_err)
    codes = np.where(live[..., None], best_codes, 0)
    scales = np.where(finite_block, best_a, POISON_SCALE)
    return codes.reshape(outer, k).astype(np.uint8), scales.astype(np.int8)


def quantize_mse_axis0(x: np.ndarray, fmt: Format, candidates: int = 4, block: int = 32):
    """quantize_mse with blocks along the rows of x: codes [cols, rows]."""
    return quantize_mse(np.ascontiguousarray(np.asarray(x).T), fmt, candidates, block)


def quantize_axis0(x: np.ndarray, fmt: Format, block: int = 32):
    """Blocks along the rows of x: quantizes x^T, giving codes [cols, rows]."""
    return quantize(np.ascontiguousarray(np.asarray(x).T), fmt, block)


def code_fields(codes: np.ndarray, fmt: Format):
    """Split element codes into (nonzero, sign, n) with n = m - B (Sec. 3.1)."""
    codes = np.asarray(codes).astype(np.int64)
    m = codes & ((1 << (fmt.E + fmt.C)) - 1)
    s = (codes >> (fmt.E + fmt.C)) & 1
    return m != 0, s, m - fmt.B


def dequantize(codes: np.ndarray, scales: np.ndarray, fmt: Format, block: int = 32) -> np.ndarray:
    """x_hat = (-1)^s 2^{a_b} r^{n/K} rounded to the nearest fp32 (Eq. curvefp-value).

    codes uint8 [outer, k] (unpacked), scales int8 [outer, k // block].
    Zero codes give +0.0; poisoned blocks (scale -128) give NaN.
    """
    codes = np.asarray(codes)
    outer, k = codes.shape
    nz, s, n = code_fields(codes, fmt)
    a = np.repeat(np.asarray(scales).astype(np.int64), block, axis=1)
    mag = np.ldexp(level_value_f64(fmt, np.where(nz, n, 0)), a)
    val = np.where(s == 1, -mag, mag)
    val = np.where(nz, val, 0.0)
    # magnitudes past the fp32 range round to +-inf, as round-to-nearest does (no warning wanted)
    with np.errstate(over="ignore"):
        out = val.astype(np.float32)
    out = np.where(a == POISON_SCALE, np.float32(np.nan), out)
    return out.astype(np.float32)


def pack7(codes: np.ndarray, block: int = 32) -> np.ndarray:
    """Pack 7-bit codes [outer, k] into [outer, k // 32, 28] bytes, LSB first."""
    codes = np.asarray(codes, dtype=np.uint8)
    assert block == 32
    outer, k = codes.shape
    assert np.all(codes < 128)
    bits = np.unpackbits(codes[..., None], axis=-1, bitorder="little")[..., :7]
    bits = bits.reshape(outer, k // 32, 32 * 7)
    return np.packbits(bits, axis=-1, bitorder="little")  # 224 bits -> 28 bytes


def unpack7(packed: np.ndarray, k: int) -> np.ndarray:
    """Inverse of pack7: [outer, k // 32, 28] bytes -> codes [outer, k]."""
    packed = np.asarray(packed, dtype=np.uint8)
    outer = packed.shape[0]
    packed = packed.reshape(outer, k // 32, 28)
    bits = np.unpackbits(packed, axis=-1, bitorder="little").reshape(outer, k // 32, 32, 7)
    weights = (1 << np.arange(7)).astype(np.uint16)
    return (bits.astype(np.uint16) * weights).sum(-1).reshape(outer, k).astype(np.uint8)


# ---------------------------------------------------------------- S-bit scale exponents

def quantize_compact(x: np.ndarray, fmt: Format, block: int, scale_bits: int):
    """Block quantization with S-bit scale exponents (Eq. effective-rate: R = 1 + E + C + S/G;
    Sec. 4.2 prices weights at S = 4 and activations at S = 5).  The paper gives only the bit
    count; the reading taken here (blocks along the rows of x):

    * each row keeps one int8 reference e_r: the largest ceil-absmax scale among its blocks that
      are finite and not all zero (0 when it has none);
    * each block keeps an unsigned S-bit offset d_b = e_r - a'_b, a'_b = max(a_b, e_r - W),
      W = 2^S - 2: a block whose own scale lies more than W below the reference is quantized at
      the raised scale a'_b (its smallest values lose resolution; nothing saturates);
    * the offset 2^S - 1 marks a block that held a NaN or an infinity (all-zero codes); an
      all-zero block has offset 0.

    Returns (codes uint8 [rows, cols], row_ref int8 [rows], offsets int64 [rows, cols // block]).
    """
    x = np.asarray(x)
    assert x.dtype == np.float32 and x.ndim == 2 and 2 <= scale_bits <= 8
    rows, cols = x.shape
    assert cols % block == 0
    nb = cols // block
    _, a = quantize(x, fmt, block)
    a = a.astype(np.int64)
    xb = x.astype(np.float64).reshape(rows, nb, block)
    finite = a != POISON_SCALE
    with np.errstate(invalid="ignore"):
        live = finite & np.any(np.where(np.isfinite(xb), xb, 0.0) != 0, axis=-1)
    ref = np.where(live.any(axis=1), np.max(np.where(live, a, SCALE_MIN - 1), axis=1), 0)
    window = (1 << scale_bits) - 2
    a_eff = np.where(live, np.maximum(a, ref[:, None] - window), ref[:, None])
    codes = np.where(live[..., None], _codes_at_scale(np.where(live[..., None], xb, 0.0), a_eff, fmt), 0)
    offsets = np.where(finite, ref[:, None] - a_eff, (1 << scale_bits) - 1)
    return codes.reshape(rows, cols).astype(np.uint8), ref.astype(np.int8), offsets


def compact_scales(row_ref: np.ndarray, offsets: np.ndarray, scale_bits: int) -> np.ndarray:
    """int8 block scales [rows, nb] of S-bit offsets: e_r - d_b, or -128 for the marker 2^S - 1."""
    ref = np.asarray(row_ref).astype(np.int64)[:, None]
    d = np.asarray(offsets).astype(np.int64)
    return np.where(d == (1 << scale_bits) - 1, POISON_SCALE, ref - d).astype(np.int8)


def pack_offsets(offsets: np.ndarray, scale_bits: int) -> np.ndarray:
    """S-bit offsets [rows, nb] packed LSB first, offset j of a row at bits [S j, S j + S) of a
    little-endian bit string, each row padded to ceil(nb S / 8) bytes."""
    d = np.asarray(offsets).astype(np.uint8)
    rows, nb = d.shape
    bits = np.unpackbits(d[..., None], axis=-1, bitorder="little")[..., :scale_bits].reshape(rows, nb * scale_bits)
    pad = (-(nb * scale_bits)) % 8
    bits = np.concatenate([bits, np.zeros((rows, pad), np.uint8)], axis=1)
    return np.packbits(bits, axis=-1, bitorder="little")


def unpack_offsets(packed: np.ndarray, nb: int, scale_bits: int) -> np.ndarray:
    """Inverse of pack_offsets."""
    p = np.asarray(packed, dtype=np.uint8)
    bits = np.unpackbits(p, axis=-1, bitorder="little")[:, : nb * scale_bits].reshape(p.shape[0], nb, scale_bits)
    return (bits.astype(np.int64) << np.arange(scale_bits)).sum(-1)


# ---------------------------------------------------------------- tensorwise scales

def quantize_tensorwise(x: np.ndarray, fmt: Format):
    """Tensorwise scale sharing (Sec. 3.1): the whole tensor is one block, quantized at the
    ceil-absmax scale of its largest magnitude.  Returns (codes uint8 [rows, cols], scales int8
    [rows, 1]): the scale repeated once per row, the rowwise layout (block = cols)."""
    x = np.asarray(x)
    assert x.dtype == np.float32 and x.ndim == 2
    rows, cols = x.shape
    codes, s = quantize(np.ascontiguousarray(x.reshape(1, rows * cols)), fmt, rows * cols)
    return codes.reshape(rows, cols), np.full((rows, 1), s[0, 0], dtype=np.int8)
