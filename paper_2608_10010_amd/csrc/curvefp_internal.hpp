// Internal declarations of libcurvefp (not part of the C ABI).
//
// Format parameters follow Sec. 3.1 / Tab. curvefp-formats of the CurveFP
// paper: E exponent bits, C curve bits, K = 2^C curves, radix r = 2^{P/Q}.  The
// flattened index n = e*K + k runs over [-(B-1), B-1] with B = 2^{E+C-1}; the
// magnitude rank is m = n + B, m = 0 is the zero sentinel, and rank m stands for
// r^{n/K} = 2^{P n / N}, N = QK (Sec. 3.2).  Binary radix is P = Q = 1.
#pragma once

#include <cstdint>
#include <hip/hip_runtime.h>

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
};

struct AllTables {
    FormatTables f[NUM_FORMATS];
};

// Builds the tables on the host.  Returns false if a self-check fails.
bool build_tables(AllTables* t);

// Per-kernel-file table upload (current device) and launchers.
hipError_t quantize_upload(const AllTables& t);
hipError_t dequantize_upload(const AllTables& t);
hipError_t gemm_upload(const AllTables& t);

// `block` (a multiple of 32 dividing the blocked extent) is the number of consecutive elements
// that share one scale in every launcher below; codes are laid out per 32 elements regardless
hipError_t launch_quantize(const void* src, int dtype, int64_t rows, int64_t cols, int64_t ld,
                           int axis, int format, int block, void* codes, int8_t* scales, hipStream_t s);
// static-operand scales: reconstruction-MSE search over `candidates` scales at or below the
// ceil-absmax scale (and, for a level pattern spanning P > 1 octaves, the P - 1 above it)
hipError_t launch_quantize_mse(const void* src, int dtype, int64_t rows, int64_t cols, int64_t ld,
                               int axis, int format, int block, int candidates, void* codes, int8_t* scales,
                               hipStream_t s);
// one scale for the whole tensor, written once per output row; workspace: one 32-bit word
hipError_t launch_quantize_tensorwise(const void* src, int dtype, int64_t rows, int64_t cols, int64_t ld, int axis,
                                     int format, void* codes, int8_t* scales, void* workspace, hipStream_t s);
// S-bit scale exponents: per row an int8 reference and packed S-bit offsets (blocks along rows)
hipError_t launch_quantize_compact(const void* src, int dtype, int64_t rows, int64_t cols, int64_t ld, int format,
                                  int block, int scale_bits, void* codes, int8_t* row_ref, uint8_t* offsets,
                                  hipStream_t s);
hipError_t launch_scales_unpack(const int8_t* row_ref, const uint8_t* offsets, int64_t rows, int64_t nblocks,
                                int scale_bits, int8_t* scales, hipStream_t s);
hipError_t launch_dequantize(const void* codes, const int8_t* scales, int format,
                             int64_t outer, int64_t k, int block, float* dst, int64_t ld_dst, hipStream_t s);
// workspace path: bytes it needs, and the launch (expansion kernels, then the GEMM)
int64_t gemm_workspace_bytes(int64_t M, int64_t N, int64_t K);
hipError_t launch_gemm_ws(const void* a, const int8_t* as, const void* b, const int8_t* bs, int64_t M,
                          int64_t N, int64_t K, int format, int block, float* c, int64_t ldc, void* ws,
                          hipStream_t s);
// curvefp_gemm_ws with C requantized in the epilogue (blocks of out_block <= 256 along each output row)
hipError_t launch_gemm_requant(const void* a, const int8_t* as, const void* b, const int8_t* bs, int64_t M, int64_t N,
                               int64_t K, int format, int block, int out_format, int out_block, void* out_codes,
                               int8_t* out_scales, void* ws, hipStream_t s);
// mixed formats / reused forward operands (trans: codes of a [K][R] tensor, blocks along R)
int64_t gemm_mixed_workspace_bytes(int64_t M, int64_t N, int64_t K);
hipError_t launch_gemm_mixed(const void* a, const int8_t* as, int fa, int ta, const void* b, const int8_t* bs, int fb,
                             int tb, int64_t M, int64_t N, int64_t K, int block, float* c, int64_t ldc, void* ws,
                             hipStream_t s);
hipError_t launch_gemm(const void* a, const int8_t* as, const void* b, const int8_t* bs,
                       int64_t M, int64_t N, int64_t K, int format, int block, float* c, int64_t ldc,
                       hipStream_t s);

}  // namespace curvefp
