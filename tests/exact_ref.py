"""Rigorous integer arithmetic used to pin the oracle (tests only).

Nothing here calls the oracle or the HIP library.  Irrational quantities
2^(v/K) are bracketed by integer K-th roots: R = floor(2^(v/K) * 2^P) =
iroot(2^(v + P*K), K), so 2^(v/K) * 2^P lies in [R, R + 1).  Every decision
below either follows from such a bracket or raises, so a silent wrong answer
is impossible.
"""

import struct
from functools import lru_cache


def iroot(n: int, k: int) -> int:
    """Largest integer r with r**k <= n (n >= 0)."""
    if n < 2:
        return n
    lo, hi = 1, 1 << (n.bit_length() // k + 1)
    while lo < hi:
        mid = (lo + hi + 1) // 2
        if mid ** k <= n:
            lo = mid
        else:
            hi = mid - 1
    return lo


@lru_cache(maxsize=None)
def frac_pow2_floor(num: int, den: int, P: int) -> int:
    """floor(2^(num/den) * 2^P) for 0 <= num <= den (num/den in lowest or any terms)."""
    assert 0 <= num <= den
    return iroot(1 << (num + P * den), den)


class Undecided(Exception):
    pass


def nearest_binary_radix(M: int, j: int, E: int, C: int, P: int = 160):
    """Nearest element of {0} U {2^(n/K)} to y = M * 2^(j-23), M in [2^23, 2^24).

    Binary radix, levels n in [-(B-1), B-1], K = 2^C, B = 2^(E+C-1).
    Returns n, or None for zero.  Raises Undecided if the bracket is too wide.
    """
    assert (1 << 23) <= M < (1 << 24)
    K = 1 << C
    B = 1 << (E + C - 1)
    n_min, n_max = -(B - 1), B - 1
    R = [frac_pow2_floor(c, K, P) for c in range(K + 1)]  # R[K] = 2^(P+1) exactly
    lhs = M << (P - 22)          # 2 y 2^(P - j)
    c_count = 0
    for c in range(K):
        S = R[c] + R[c + 1]      # (2^(c/K) + 2^((c+1)/K)) 2^P in [S, S + 2)
        if lhs >= S + 2:
            c_count += 1
        elif lhs <= S:
            pass                  # the sum is irrational, so lhs < true threshold
        else:
            raise Undecided((M, j, c))
    n = K * j + c_count
    if n > n_max:
        return n_max
    if n >= n_min:
        return n
    # zero or n_min: compare 2y with 2^(n_min/K) = 2^e0 * 2^(k0/K)
    e0, k0 = divmod(n_min, K)
    assert k0 != 0
    shift = j - 22 - e0 + P
    assert shift >= 0
    lhs2 = M << shift             # 2y * 2^(P - e0)
    Rk = frac_pow2_floor(k0, K, P)
    if lhs2 >= Rk + 1:
        return n_min
    if lhs2 <= Rk:
        return None
    raise Undecided((M, j, "zero"))


def rn_f32_pow2(a: int, n: int, K: int, P: int = 200) -> float:
    """Nearest float32 (ties to even) to 2^(a + n/K), decided rigorously."""
    return rn_f32_level(a, n, 1, K, P)


def rn_f32_level(a: int, n: int, p: int, N: int, P: int = 200) -> float:
    """Nearest float32 (ties to even) to 2^(a + p n / N), decided rigorously."""
    e, k = divmod(p * n, N)
    K = N
    Ex = a + e                    # value = 2^Ex * 2^(k/K)
    if k == 0:
        if Ex > 127:
            return float("inf")
        if Ex >= -149:
            return 2.0 ** Ex
        return 0.0                # 2^-150 ties to even (zero); smaller rounds to zero
    R = frac_pow2_floor(k, K, P)  # 2^(k/K) 2^P in (R, R + 1)
    if Ex >= -126:
        keep = 23                 # significand bits below the leading one
        lo_exp = Ex
    else:
        keep = 23 - (-126 - Ex)   # subnormal: unit is 2^-149
        lo_exp = -126
        if keep < -1:
            return 0.0
    # q = round(2^(k/K) * 2^keep); value = q * 2^(Ex - keep)
    def rnd(x_scaled):            # x_scaled = integer approx of 2^(k/K) * 2^P
        sh = P - keep
        q, r = divmod(x_scaled, 1 << sh)
        half = 1 << (sh - 1)
        return q + (1 if r > half else 0), r == half
    q0, t0 = rnd(R)
    q1, t1 = rnd(R + 1)
    if q0 != q1 or t0 or t1:
        # the true value lies strictly between R and R + 1; disagreement means undecided
        if q0 != q1:
            raise Undecided((a, n))
    q = q0
    val = q * 2.0 ** (Ex - keep)
    if val >= 2.0 ** 128:
        return float("inf")
    return struct.unpack("<f", struct.pack("<f", val))[0]


def f32_bits(x: float) -> int:
    return struct.unpack("<I", struct.pack("<f", x))[0]


# ---------------------------------------------------------------- rational radix r = 2^(p/q)

class Tie(Exception):
    """y sits exactly on a decision point (possible only where the point is dyadic)."""


def _level_parts(n: int, p: int, N: int):
    """2^(p n / N) = 2^w * 2^(r / N), 0 <= r < N."""
    return divmod(p * n, N)


def _above_midpoint(M: int, j: int, n: int, p: int, N: int, P: int) -> bool:
    """y = M 2^(j-23) > (L(n) + L(n+1)) / 2, L(n) = 2^(p n / N), decided with brackets
    F(r) = floor(2^(r/N) 2^P), exact only for r = 0."""
    w0, r0 = _level_parts(n, p, N)
    w1, r1 = _level_parts(n + 1, p, N)
    d = w1 - w0
    assert d >= 0
    S = frac_pow2_floor(r0, N, P) + (frac_pow2_floor(r1, N, P) << d)
    width = (0 if r0 == 0 else 1) + (0 if r1 == 0 else (1 << d))
    sh = j - 22 + P - w0
    assert sh >= 0
    lhs = M << sh                                  # 2 y 2^(P - w0)
    if width == 0:
        if lhs == S:
            raise Tie((M, j, n))
        return lhs > S
    if lhs >= S + width:
        return True
    if lhs <= S:
        return False
    raise Undecided((M, j, n))


def nearest_level(M: int, j: int, E: int, C: int, p: int, q: int, P: int = 240):
    """Nearest element of {0} U {2^(p n / N)}, N = qK, to y = M 2^(j-23), M in [2^23, 2^24),
    levels n in [-(B-1), B-1].  Returns n, or None for zero.  A tie between zero and the smallest
    level (possible when its half is dyadic) goes to the level, the reading the library takes.
    Raises Undecided if a bracket is too wide."""
    assert (1 << 23) <= M < (1 << 24)
    K = 1 << C
    N = q * K
    B = 1 << (E + C - 1)
    n_min, n_max = -(B - 1), B - 1
    # midpoints increase with n: the nearest level is n_min + #{n : y above midpoint n}
    lo, hi = n_min, n_max            # find the count by bisection over the monotone predicate
    while lo < hi:
        mid = (lo + hi) // 2
        if _above_midpoint(M, j, mid, p, N, P):
            lo = mid + 1
        else:
            hi = mid
    n = lo
    if n > n_min:
        return n
    # zero or n_min: 2y against L(n_min)
    w, r = _level_parts(n_min, p, N)
    sh = j - 22 + P - w
    assert sh >= 0
    lhs = M << sh                    # 2 y 2^(P - w)
    F = frac_pow2_floor(r, N, P)
    if r == 0:
        return n_min if lhs >= F else None     # lhs == F: the tie, to the level
    if lhs >= F + 1:
        return n_min
    if lhs <= F:
        return None
    raise Undecided((M, j, "zero"))
