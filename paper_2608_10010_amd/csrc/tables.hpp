// Format constants of CurveFP and the layout of libcurvefp's constant tables.  Host-only (no
// HIP): the table generator, built and run before the kernels are compiled, includes it too.
//
// Format parameters follow Sec. 3.1 / Tab. curvefp-formats of the CurveFP
// paper: E exponent bits, C curve bits, K = 2^C curves, radix r = 2^{P/Q}.  The
// flattened index n = e*K + k runs over [-(B-1), B-1] with B = 2^{E+C-1}; the
// magnitude rank is m = n + B, m = 0 is the zero sentinel, and rank m stands for
// r^{n/K} = 2^{P n / N}, N = QK (Sec. 3.2).  Binary radix is P = Q = 1.
#pragma once

#include <cstdint>

namespace curvefp {

constexpr int floor_div_c(int a, int b) { return a / b - ((a % b != 0) && ((a < 0) != (b < 0)) ? 1 : 0); }
constexpr int gcd_c(int a, int b) { return b == 0 ? a : gcd_c(b, a % b); }

template <int E_, int C_, int P_ = 1, int Q_ = 1>
struct Fmt {
    static constexpr int E = E_;
    static constexpr int C = C_;
    static constexpr int P = P_;
    static constexpr int Q = Q_;
    static constexpr int K = 1 << C;
    static constexpr int N = Q * K;                 // exponent residues: 2^{P n / N}
    static constexpr bool BINARY = P == 1 && Q == 1;
    // octaves after which the level pattern repeats (2^{P'} = r^{N'/K} in lowest terms)
    static constexpr int PERIOD = P / gcd_c(P, N);
    static constexpr int EC = E + C;
    static constexpr int B = 1 << (EC - 1);
    static constexpr int NMAX = B - 1;
    static constexpr int NMIN = -(B - 1);
    static constexpr int MAG_MASK = (1 << EC) - 1;
    static constexpr int NMAG = 1 << EC;            // magnitude ranks 0 .. 2^{E+C}-1
    static constexpr bool PACKED7 = (EC + 1) == 7;  // E3C3 codes are 7 bits
    // octave of the smallest level's zero threshold 2^{P n_min / N - 1}, and of the top level
    static constexpr int OZ = floor_div_c(P * NMIN - N, N);
    static constexpr int OHI = floor_div_c(P * NMAX, N);
    // quantize table: one entry per bf16-truncated magnitude in octaves [OZ, OHI]
    static constexpr int QLUT_SIZE = (OHI - OZ + 1) * 128;
    // below this scale, subnormal inputs can reach a nonzero code and need exact normalization
    static constexpr int A_FAST_MIN = -126 - OZ;
    // GEMM decode: fp16 exponent bias so that the largest element of a row lands near 2^15
    static constexpr int GEMM_BIAS = 15 - OHI;
};

using FmtE4C3 = Fmt<4, 3>;
using FmtE5C2 = Fmt<5, 2>;
using FmtE3C3 = Fmt<3, 3>;
// the E4C3 radices of Tab. radix-frontier: r = 2^{8/9} (9 phases), r = 2^{3/4} (32 phases)
using FmtE4C3R89 = Fmt<4, 3, 8, 9>;
using FmtE4C3R34 = Fmt<4, 3, 3, 4>;

// format ids of the C ABI (curvefp_format) index the tables
constexpr int NUM_FORMATS = 5;

static_assert(FmtE4C3::OZ == -9 && FmtE5C2::OZ == -17 && FmtE3C3::OZ == -5, "zero-threshold octaves");
static_assert(FmtE4C3::OHI == 7 && FmtE5C2::OHI == 15 && FmtE3C3::OHI == 3, "top octaves");
static_assert(FmtE4C3R89::OZ == -8 && FmtE4C3R89::OHI == 7, "2^(8/9): levels 2^(n/9), 2^-7 .. 2^7");
static_assert(FmtE4C3R34::OZ == -7 && FmtE4C3R34::OHI == 5, "2^(3/4): levels 2^(3n/32), 2^-5.9 .. 2^5.9");
static_assert(FmtE4C3::PERIOD == 1 && FmtE4C3R89::PERIOD == 1 && FmtE4C3R34::PERIOD == 3, "pattern periods");

// GEMM expansion table: one (lo16 << 16) | hi16 fp16 pair per code byte (sign included),
// for a block whose scale equals its row's largest; other blocks are scaled by 2^-D in fp16.
constexpr int GEMM_DEC_ENTRIES = 256;

constexpr int QLUT_MAX = FmtE5C2::QLUT_SIZE;   // the largest of the formats'

// Host-built constant tables for one format (long double arithmetic, own derivation).
struct FormatTables {
    int K = 0;
    int P = 1, Q = 1;               // radix 2^{P/Q}
    int qlut_size = 0;
    uint32_t qlut[QLUT_MAX];        // (m_base << 16) | thr16, see quantize.hip
    uint32_t lmax_mant = 0;         // mantissa field of fl32 of the top level
    uint32_t mant[8];               // binary radix: mantissa field of fl32(2^{k/K}), k < K
    uint64_t sig62[8];              // binary radix: floor(2^{k/K} * 2^62)
    uint32_t dq_em[128];            // per magnitude rank: (w << 24) | mantissa of fl32(2^{f/N}),
    uint64_t dq_sig62[128];         //   floor(2^{f/N} 2^62), for 2^{P n / N} = 2^{w + f/N}
    uint32_t dec[GEMM_DEC_ENTRIES];  // (lo16 << 16) | hi16 fp16 pair per code byte
    // the decision points of the nearest-level rule, for the generator's report: point i lies
    // between levels nmin + i and nmin + i + 1 as (octave, 24-bit significand threshold); a
    // magnitude M 2^{o-23} is above it iff (o, M) > (point_o, point_T)
    int npoints = 0;
    int point_o[256];
    int64_t point_T[256];
    int zero_o = 0;                 // half the smallest level, as a point of the same kind
    int64_t zero_T = 0;
    int zero_exact = 0;             // the zero point is a float itself (a tie goes to the level)
};

struct AllTables {
    FormatTables f[NUM_FORMATS];
};

// Builds the tables on the host (the build's table generator calls it; the library holds the
// result as compile-time constants).  Returns false if a self-check fails.
bool build_tables(AllTables* t);

}  // namespace curvefp
