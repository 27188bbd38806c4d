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

#include "tables.hpp"

namespace curvefp {


// Launchers (the constant tables are compile-time __constant__ arrays of each kernel file).

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
// quantize [rows][k] along k and write the result's prepared form (launch_prepare's layout, trans 0)
// and, if dst is not null, its reconstruction; block in 32..512 (a power of two), k % block == 0
hipError_t launch_quantize_prepare(const void* src, int dtype, int64_t rows, int64_t k, int64_t ld, int format,
                                  int block, void* codes, int8_t* scales, void* prepared, float* dst, int64_t ld_dst,
                                  hipStream_t s);
// the same for the two operands of one GEMM (same k, dtype, format and block) in one launch
hipError_t launch_quantize_prepare_pair(const void* src_a, int64_t rows_a, int64_t ld_a, void* codes_a,
                                       int8_t* scales_a, void* prepared_a, float* dst_a, int64_t ld_dst_a,
                                       const void* src_b, int64_t rows_b, int64_t ld_b, void* codes_b,
                                       int8_t* scales_b, void* prepared_b, float* dst_b, int64_t ld_dst_b, int dtype,
                                       int64_t k, int format, int block, hipStream_t s);
hipError_t launch_dequantize(const void* codes, const int8_t* scales, int format,
                             int64_t outer, int64_t k, int block, float* dst, int64_t ld_dst, hipStream_t s);
// workspace path: bytes it needs, and the launch (expansion kernels, then the GEMM)
int64_t gemm_workspace_bytes(int64_t M, int64_t N, int64_t K);
hipError_t launch_gemm_ws(const void* a, const int8_t* as, const void* b, const int8_t* bs, int64_t M,
                          int64_t N, int64_t K, int format, int block, float* c, int64_t ldc, void* ws,
                          hipStream_t s);
// prepared operands: one operand's expansion (planes + row maxima), and the GEMM on two of them
int64_t prepared_bytes(int64_t rows, int64_t K, int trans);
int64_t gemm_prepared_workspace_bytes(int64_t M, int64_t N, int64_t K);
hipError_t launch_prepare(const void* codes, const int8_t* scales, int64_t rows, int64_t K, int format, int block,
                          int trans, void* prepared, hipStream_t s);
hipError_t launch_gemm_prepared(const void* pa, int fa, const void* pb, int fb, int64_t M, int64_t N, int64_t K,
                                float* c, int64_t ldc, void* ws, hipStream_t s);
// curvefp_gemm_ws with C requantized in the epilogue (blocks of out_block <= 256 along each output row)
hipError_t launch_gemm_requant(const void* a, const int8_t* as, const void* b, const int8_t* bs, int64_t M, int64_t N,
                               int64_t K, int format, int block, int out_format, int out_block, void* out_codes,
                               int8_t* out_scales, void* ws, hipStream_t s);
// mixed formats / reused forward operands (trans: codes of a [K][R] tensor, blocks along R)
int64_t gemm_mixed_workspace_bytes(int64_t M, int64_t N, int64_t K);
hipError_t launch_gemm_mixed(const void* a, const int8_t* as, int fa, int ta, const void* b, const int8_t* bs, int fb,
                             int tb, int64_t M, int64_t N, int64_t K, int block, float* c, int64_t ldc, void* ws,
                             hipStream_t s);
// the calling device's static scratch (CURVEFP_STATIC_SCRATCH_BYTES, 256-byte aligned), looked up
// on the device's first call and kept
hipError_t static_scratch(void** out);
hipError_t launch_gemm(const void* a, const int8_t* as, const void* b, const int8_t* bs,
                       int64_t M, int64_t N, int64_t K, int format, int block, float* c, int64_t ldc,
                       hipStream_t s);

}  // namespace curvefp
