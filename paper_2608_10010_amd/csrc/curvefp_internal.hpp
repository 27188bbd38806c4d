// Internal declarations of libcurvefp (not part of the C ABI).
//
// Format parameters follow Sec. 3.1 / Tab. curvefp-formats of the CurveFP
// paper: E exponent bits, C curve bits, K = 2^C curves, binary radix.  The
// flattened index n = e*K + k runs over [-(B-1), B-1] with B = 2^{E+C-1};
// the magnitude rank is m = n + B and m = 0 is the zero sentinel.
#pragma once

#include <cstdint>
#include <hip/hip_runtime.h>

namespace curvefp {

template <int E_, int C_>
struct Fmt {
    static constexpr int E = E_;
    static constexpr int C = C_;
    static constexpr int K = 1 << C;
    static constexpr int EC = E + C;
    static constexpr int B = 1 << (EC - 1);
    static constexpr int NMAX = B - 1;
    static constexpr int NMIN = -(B - 1);
    static constexpr int MAG_MASK = (1 << EC) - 1;
    static constexpr int NMAG = 1 << EC;            // magnitude ranks 0 .. 2^{E+C}-1
    static constexpr bool PACKED7 = (EC + 1) == 7;  // E3C3 codes are 7 bits
    // octave of the smallest level's zero threshold 2^{n_min/K - 1}, and of the top level
    static constexpr int OZ = (NMIN - K) / K - ((NMIN - K) % K != 0 ? 1 : 0);  // floor((n_min - K) / K)
    static constexpr int OHI = NMAX / K;                                       // floor(n_max / K), n_max > 0
    static constexpr int EMAX = (1 << (E - 1)) - 1;   // largest element exponent e
    // quantize table: one entry per bf16-truncated magnitude in octaves [OZ, OHI]
    static constexpr int QLUT_SIZE = (OHI - OZ + 1) * 128;
    // below this scale, subnormal inputs can reach a nonzero code and need exact normalization
    static constexpr int A_FAST_MIN = -126 - OZ;
    // GEMM decode: fp16 exponent bias so that the largest element of a row lands near 2^15
    static constexpr int GEMM_BIAS = 15 - EMAX;
};

using FmtE4C3 = Fmt<4, 3>;
using FmtE5C2 = Fmt<5, 2>;
using FmtE3C3 = Fmt<3, 3>;

static_assert(FmtE4C3::OZ == -9 && FmtE5C2::OZ == -17 && FmtE3C3::OZ == -5, "zero-threshold octaves");
static_assert(FmtE4C3::OHI == 7 && FmtE5C2::OHI == 15 && FmtE3C3::OHI == 3, "top octaves");

// GEMM expansion table: one (lo16 << 16) | hi16 fp16 pair per code byte (sign included),
// for a block whose scale equals its row's largest; other blocks are scaled by 2^-D in fp16.
constexpr int GEMM_DEC_ENTRIES = 256;

constexpr int QLUT_MAX = FmtE5C2::QLUT_SIZE;   // largest of the three

// Host-built constant tables for one format (long double arithmetic, own derivation).
struct FormatTables {
    int K = 0;
    int qlut_size = 0;
    uint32_t qlut[QLUT_MAX];        // (m_base << 16) | thr16, see quantize.hip
    uint32_t lmax_mant = 0;         // mantissa field of fl32(2^{(K-1)/K})
    uint32_t mant[8];               // mantissa field of fl32(2^{k/K}), k < K
    uint64_t sig62[8];              // floor(2^{k/K} * 2^62)
    uint32_t dec[GEMM_DEC_ENTRIES];  // (lo16 << 16) | hi16 fp16 pair per code byte
};

struct AllTables {
    FormatTables f[3];
};

// Builds the tables on the host.  Returns false if a self-check fails.
bool build_tables(AllTables* t);

// Per-kernel-file table upload (current device) and launchers.
hipError_t quantize_upload(const AllTables& t);
hipError_t dequantize_upload(const AllTables& t);
hipError_t gemm_upload(const AllTables& t);

hipError_t launch_quantize(const void* src, int dtype, int64_t rows, int64_t cols, int64_t ld,
                           int axis, int format, void* codes, int8_t* scales, hipStream_t s);
hipError_t launch_dequantize(const void* codes, const int8_t* scales, int format,
                             int64_t outer, int64_t k, float* dst, int64_t ld_dst, hipStream_t s);
// workspace path: bytes it needs, and the launch (expansion kernels, then the GEMM)
int64_t gemm_workspace_bytes(int64_t M, int64_t N, int64_t K);
hipError_t launch_gemm_ws(const void* a, const int8_t* as, const void* b, const int8_t* bs, int64_t M,
                          int64_t N, int64_t K, int format, float* c, int64_t ldc, void* ws, hipStream_t s);
// mixed formats / reused forward operands (trans: codes of a [K][R] tensor, blocks along R)
int64_t gemm_mixed_workspace_bytes(int64_t M, int64_t N, int64_t K);
hipError_t launch_gemm_mixed(const void* a, const int8_t* as, int fa, int ta, const void* b, const int8_t* bs, int fb,
                             int tb, int64_t M, int64_t N, int64_t K, float* c, int64_t ldc, void* ws, hipStream_t s);
hipError_t launch_gemm(const void* a, const int8_t* as, const void* b, const int8_t* bs,
                       int64_t M, int64_t N, int64_t K, int format, float* c, int64_t ldc,
                       hipStream_t s);

}  // namespace curvefp
