"""CurveFP format parameters (oracle side; test infrastructure only).

A format is the tuple (E, C, p/q) of Sec. 3.1: E exponent bits, C curve-index
bits, K = 2**C curves, and radix r = 2**(p/q).  A nonzero element is
(-1)^s * 2^{a_b} * r^{e + k/K} with e in [-2^{E-1}, 2^{E-1}-1] and k in [0, K)
(Eq. curvefp-value).  The flattened index n = e*K + k (Sec. 2 "Logarithmic
neural-network arithmetic", Sec. 3.2) therefore runs over [-B, B-1] with
B = 2^{E+C-1}.  The paper reserves magnitude index zero as the zero sentinel
and drops the smallest nonzero exponent/curve combination, n = -B, leaving
2^{E+C} - 1 positive magnitudes n in [-(B-1), B-1] (Sec. 3.1, Tab.
curvefp-formats).

Element code (reading of Sec. 3.1 together with the tile encoding of App. C.1,
where the sign sits in the top bit, the magnitude rank m in the low E+C bits,
m = 0 is zero and q = m - 64 for E4C3):  code = s << (E+C) | m, m = n + B.
"""

from dataclasses import dataclass
from math import gcd


@dataclass(frozen=True)
class Format:
    name: str
    E: int          # exponent field width
    C: int          # curve-index field width
    p: int = 1      # radix r = 2^(p/q)  (p = q = 1: binary radix)
    q: int = 1

    @property
    def K(self) -> int:
        """Number of interleaved curves, K = 2^C (Sec. 3.1)."""
        return 2 ** self.C

    @property
    def B(self) -> int:
        """Offset between the flattened index n and the magnitude rank m."""
        return 2 ** (self.E + self.C - 1)

    @property
    def n_min(self) -> int:
        return -(self.B - 1)

    @property
    def n_max(self) -> int:
        return self.B - 1

    @property
    def bits(self) -> int:
        """Element width 1 + E + C (Sec. 3.1)."""
        return 1 + self.E + self.C

    @property
    def positive_levels(self) -> int:
        return self.n_max - self.n_min + 1

    @property
    def N(self) -> int:
        """N = qK, the modulus of the fractional-exponent residue (Sec. 3.2)."""
        return self.q * self.K

    @property
    def g(self) -> int:
        return gcd(self.p, self.N)

    @property
    def H(self) -> int:
        """Phase count H = qK / gcd(p, qK) (Eq. phase-count)."""
        return self.N // self.g

    def storage_rate(self, G: int, S: int) -> float:
        """Bits per value R = 1 + E + C + S/G (Eq. effective-rate)."""
        return self.bits + S / G


def rational_format(E: int, C: int, p: int, q: int) -> Format:
    """A format with rational radix r = 2^(p/q) (Sec. 3.1, Tab. radix-frontier)."""
    return Format(f"E{E}C{C}_r{p}/{q}", E, C, p, q)


# Tab. curvefp-formats: CurveFP7 E3C3, CurveFP8 E4C3 / E5C2, all binary radix; and the two
# E4C3 radices of Tab. radix-frontier, r = 2^(8/9) (9 phases) and r = 2^(3/4) (32 phases).
FORMATS = {
    "E4C3": Format("E4C3", 4, 3),
    "E5C2": Format("E5C2", 5, 2),
    "E3C3": Format("E3C3", 3, 3),
    "E4C3_r8/9": rational_format(4, 3, 8, 9),
    "E4C3_r3/4": rational_format(4, 3, 3, 4),
}


def get_format(name: str) -> Format:
    return FORMATS[name]
