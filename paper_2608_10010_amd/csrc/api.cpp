// C ABI of libcurvefp: argument validation and dispatch.
// Validation runs before any HIP call, so every argument error is reported
// without touching the device.  The library keeps no state: its constant tables
// are compile-time __constant__ arrays of the kernel files, and a call does
// nothing but validate its arguments and launch on the caller's stream.

#include "../../include/curvefp.h"
#include "curvefp_internal.hpp"

using namespace curvefp;

namespace {

// per format id: element bits, E, C, radix r = 2^{P/Q}
constexpr int kBits[NUM_FORMATS] = {8, 8, 7, 8, 8};
constexpr int kE[NUM_FORMATS] = {4, 5, 3, 4, 4};
constexpr int kC[NUM_FORMATS] = {3, 2, 3, 3, 3};
constexpr int kP[NUM_FORMATS] = {1, 1, 1, 8, 3};
constexpr int kQ[NUM_FORMATS] = {1, 1, 1, 9, 4};

bool fmt_ok(int f) { return f >= 0 && f < NUM_FORMATS; }

// elements per scale: a positive multiple of 32 (codes stay laid out per 32 elements)
bool block_ok(int b) { return b >= 32 && b % 32 == 0 && b <= (1 << 30); }

int gcd_i(int a, int b) {
    while (b) {
        const int r = a % b;
        a = b;
        b = r;
    }
    return a;
}
bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int hip_status(hipError_t e) { return e == hipSuccess ? CURVEFP_OK : CURVEFP_ERR_HIP; }

// contraction length of the GEMM entry points: positive, whole groups of 32, at most CURVEFP_MAX_K
bool gemm_k_ok(int64_t K) { return K > 0 && K % 32 == 0 && K <= CURVEFP_MAX_K; }

// one operand of curvefp_quantize_prepare(_pair): the status of its arguments
int qp_check(int dtype, int64_t k, int format, int block, const void* src, int64_t rows, int64_t ld_src,
             const void* codes, const int8_t* scales, const void* prepared, int64_t prepared_size, const float* dst,
             int64_t ld_dst) {
    if (!src || !codes || !scales || !prepared) return CURVEFP_ERR_NULL;
    if ((dtype != 0 && dtype != 1) || !fmt_ok(format)) return CURVEFP_ERR_FORMAT;
    // a block's maximum is reduced over the 4 .. 64 lanes that hold it
    if (block != 32 && block != 64 && block != 128 && block != 256 && block != 512) return CURVEFP_ERR_BLOCK;
    if (rows <= 0 || rows >= ((int64_t)1 << 31) || k <= 0 || k % block || ld_src < k) return CURVEFP_ERR_SHAPE;
    if (k > CURVEFP_MAX_K) return CURVEFP_ERR_SHAPE;   // the prepared form's bound
    if (dst && ld_dst < k) return CURVEFP_ERR_SHAPE;
    if (prepared_size < prepared_bytes(rows, k, 0)) return CURVEFP_ERR_SHAPE;
    const int64_t esz = dtype == 1 ? 2 : 4;
    if (!aligned16(src) || (ld_src * esz) % 16 || !aligned16(codes) || reinterpret_cast<uintptr_t>(prepared) % 256)
        return CURVEFP_ERR_ALIGN;
    if (dst && (!aligned16(dst) || (ld_dst * 4) % 16)) return CURVEFP_ERR_ALIGN;
    return CURVEFP_OK;
}

}  // namespace

#pragma GCC visibility push(default)
extern "C" {

int curvefp_format_info(int format, int* bits, int* E, int* C, int* phases) {
    if (!fmt_ok(format)) return CURVEFP_ERR_FORMAT;
    if (bits) *bits = kBits[format];
    if (E) *E = kE[format];
    if (C) *C = kC[format];
    const int qk = kQ[format] << kC[format];
    if (phases) *phases = qk / gcd_i(kP[format], qk);   // H = qK / gcd(p, qK)
    return CURVEFP_OK;
}

int curvefp_format_radix(int format, int* p, int* q) {
    if (!fmt_ok(format)) return CURVEFP_ERR_FORMAT;
    if (p) *p = kP[format];
    if (q) *q = kQ[format];
    return CURVEFP_OK;
}

int64_t curvefp_codes_bytes(int format, int64_t outer, int64_t k, int block) {
    if (!fmt_ok(format)) return CURVEFP_ERR_FORMAT;
    if (!block_ok(block)) return CURVEFP_ERR_BLOCK;
    if (outer < 0 || k < 0 || k % block) return CURVEFP_ERR_SHAPE;
    return format == CURVEFP_E3C3 ? outer * (k / 32) * 28 : outer * k;
}

int64_t curvefp_scales_count(int64_t outer, int64_t k, int block) {
    if (!block_ok(block)) return CURVEFP_ERR_BLOCK;
    if (outer < 0 || k < 0 || k % block) return CURVEFP_ERR_SHAPE;
    return outer * (k / block);
}

int curvefp_quantize(const void* src, int dtype, int64_t rows, int64_t cols, int64_t ld_src,
                     int block_axis, int format, int block, void* codes, int8_t* scales,
                     void* stream) {
    if (!src || !codes || !scales) return CURVEFP_ERR_NULL;
    if (!fmt_ok(format) || (dtype != CURVEFP_F32 && dtype != CURVEFP_BF16)) return CURVEFP_ERR_FORMAT;
    if (!block_ok(block) || (block_axis != 0 && block_axis != 1)) return CURVEFP_ERR_BLOCK;
    if (rows <= 0 || cols <= 0 || ld_src < cols) return CURVEFP_ERR_SHAPE;
    if ((block_axis == 1 ? cols : rows) % block) return CURVEFP_ERR_SHAPE;
    const int esz = dtype == CURVEFP_F32 ? 4 : 2;
    // blocks along rows are read with 16-byte vector loads; the transpose path reads elements
    if (!aligned16(codes)) return CURVEFP_ERR_ALIGN;
    if (block_axis == 1 && (!aligned16(src) || (ld_src * esz) % 16)) return CURVEFP_ERR_ALIGN;
    if (block_axis == 0 && (reinterpret_cast<uintptr_t>(src) % esz)) return CURVEFP_ERR_ALIGN;
    return hip_status(launch_quantize(src, dtype, rows, cols, ld_src, block_axis, format, block, codes, scales,
                                      reinterpret_cast<hipStream_t>(stream)));
}

int curvefp_quantize_tensorwise(const void* src, int dtype, int64_t rows, int64_t cols, int64_t ld_src,
                                int block_axis, int format, void* codes, int8_t* scales, void* workspace,
                                void* stream) {
    if (!src || !codes || !scales || !workspace) return CURVEFP_ERR_NULL;
    if (!fmt_ok(format) || (dtype != CURVEFP_F32 && dtype != CURVEFP_BF16)) return CURVEFP_ERR_FORMAT;
    if (block_axis != 0 && block_axis != 1) return CURVEFP_ERR_BLOCK;
    if (rows <= 0 || cols <= 0 || ld_src < cols) return CURVEFP_ERR_SHAPE;
    if ((block_axis == 1 ? cols : rows) % 32 || (block_axis == 1 ? cols : rows) > (1 << 30)) return CURVEFP_ERR_SHAPE;
    if (rows >= ((int64_t)1 << 31) || cols >= ((int64_t)1 << 31)) return CURVEFP_ERR_SHAPE;
    const int esz = dtype == CURVEFP_F32 ? 4 : 2;
    if (!aligned16(codes) || (reinterpret_cast<uintptr_t>(workspace) & 3)) return CURVEFP_ERR_ALIGN;
    if (block_axis == 1 && (!aligned16(src) || (ld_src * esz) % 16)) return CURVEFP_ERR_ALIGN;
    if (block_axis == 0 && (reinterpret_cast<uintptr_t>(src) % esz)) return CURVEFP_ERR_ALIGN;
    return hip_status(launch_quantize_tensorwise(src, dtype, rows, cols, ld_src, block_axis, format, codes, scales,
                                                 workspace, reinterpret_cast<hipStream_t>(stream)));
}

int64_t curvefp_compact_offsets_bytes(int64_t rows, int64_t cols, int block, int scale_bits) {
    if (!block_ok(block) || scale_bits < 2 || scale_bits > 8) return CURVEFP_ERR_BLOCK;
    if (rows < 0 || cols < 0 || cols % block) return CURVEFP_ERR_SHAPE;
    return rows * ((cols / block * scale_bits + 7) / 8);
}

int curvefp_quantize_compact(const void* src, int dtype, int64_t rows, int64_t cols, int64_t ld_src, int format,
                             int block, int scale_bits, void* codes, int8_t* row_ref, uint8_t* offsets,
                             void* stream) {
    if (!src || !codes || !row_ref || !offsets) return CURVEFP_ERR_NULL;
    if (!fmt_ok(format) || (dtype != CURVEFP_F32 && dtype != CURVEFP_BF16)) return CURVEFP_ERR_FORMAT;
    if (!block_ok(block) || scale_bits < 2 || scale_bits > 8) return CURVEFP_ERR_BLOCK;
    if (rows <= 0 || cols <= 0 || ld_src < cols || cols % block) return CURVEFP_ERR_SHAPE;
    if (cols > 131072 || rows > 0x7FFFFFFF) return CURVEFP_ERR_SHAPE;   // one workgroup per row
    const int esz = dtype == CURVEFP_F32 ? 4 : 2;
    if (!aligned16(codes) || !aligned16(src) || (ld_src * esz) % 16) return CURVEFP_ERR_ALIGN;
    return hip_status(launch_quantize_compact(src, dtype, rows, cols, ld_src, format, block, scale_bits, codes,
                                              row_ref, offsets, reinterpret_cast<hipStream_t>(stream)));
}

int curvefp_scales_unpack(const int8_t* row_ref, const uint8_t* offsets, int64_t rows, int64_t nblocks,
                          int scale_bits, int8_t* scales, void* stream) {
    if (!row_ref || !offsets || !scales) return CURVEFP_ERR_NULL;
    if (scale_bits < 2 || scale_bits > 8) return CURVEFP_ERR_BLOCK;
    if (rows <= 0 || nblocks <= 0 || rows * nblocks >= ((int64_t)1 << 39)) return CURVEFP_ERR_SHAPE;
    return hip_status(launch_scales_unpack(row_ref, offsets, rows, nblocks, scale_bits, scales,
                                           reinterpret_cast<hipStream_t>(stream)));
}

int curvefp_quantize_mse(const void* src, int dtype, int64_t rows, int64_t cols, int64_t ld_src,
                         int block_axis, int format, int block, int candidates, void* codes, int8_t* scales,
                         void* stream) {
    if (!src || !codes || !scales) return CURVEFP_ERR_NULL;
    if (!fmt_ok(format) || (dtype != CURVEFP_F32 && dtype != CURVEFP_BF16)) return CURVEFP_ERR_FORMAT;
    if (!block_ok(block) || (block_axis != 0 && block_axis != 1)) return CURVEFP_ERR_BLOCK;
    if (candidates < 1 || candidates > 8) return CURVEFP_ERR_SHAPE;
    if (rows <= 0 || cols <= 0 || ld_src < cols) return CURVEFP_ERR_SHAPE;
    if ((block_axis == 1 ? cols : rows) % block) return CURVEFP_ERR_SHAPE;
    if (rows * cols / 32 / 256 >= ((int64_t)1 << 31)) return CURVEFP_ERR_SHAPE;
    const int esz = dtype == CURVEFP_F32 ? 4 : 2;
    if (!aligned16(codes)) return CURVEFP_ERR_ALIGN;
    if (block_axis == 1 && (!aligned16(src) || (ld_src * esz) % 16)) return CURVEFP_ERR_ALIGN;
    if (block_axis == 0 && (reinterpret_cast<uintptr_t>(src) % esz)) return CURVEFP_ERR_ALIGN;
    return hip_status(launch_quantize_mse(src, dtype, rows, cols, ld_src, block_axis, format, block, candidates, codes,
                                          scales,
                                          reinterpret_cast<hipStream_t>(stream)));
}

int curvefp_dequantize(const void* codes, const int8_t* scales, int format, int64_t outer, int64_t k,
                       int block, float* dst, int64_t ld_dst, void* stream) {
    if (!codes || !scales || !dst) return CURVEFP_ERR_NULL;
    if (!fmt_ok(format)) return CURVEFP_ERR_FORMAT;
    if (!block_ok(block)) return CURVEFP_ERR_BLOCK;
    if (outer <= 0 || k <= 0 || k % block || ld_dst < k) return CURVEFP_ERR_SHAPE;
    if (!aligned16(codes) || !aligned16(dst) || (ld_dst * 4) % 16) return CURVEFP_ERR_ALIGN;
    return hip_status(launch_dequantize(codes, scales, format, outer, k, block, dst, ld_dst,
                                        reinterpret_cast<hipStream_t>(stream)));
}

int curvefp_gemm(const void* a_codes, const int8_t* a_scales, const void* b_codes, const int8_t* b_scales,
                 int64_t M, int64_t N, int64_t K, int format, int block, float* c, int64_t ldc,
                 void* stream) {
    if (!a_codes || !a_scales || !b_codes || !b_scales || !c) return CURVEFP_ERR_NULL;
    if (!fmt_ok(format)) return CURVEFP_ERR_FORMAT;
    if (!block_ok(block)) return CURVEFP_ERR_BLOCK;
    if (M <= 0 || N <= 0 || !gemm_k_ok(K) || K % block || ldc < N) return CURVEFP_ERR_SHAPE;
    if (M > CURVEFP_MAX_M_FUSED) return CURVEFP_ERR_SHAPE;
    if (!aligned16(a_codes) || !aligned16(b_codes) || !aligned16(c)) return CURVEFP_ERR_ALIGN;
    return hip_status(launch_gemm(a_codes, a_scales, b_codes, b_scales, M, N, K, format, block, c, ldc,
                                  reinterpret_cast<hipStream_t>(stream)));
}

int64_t curvefp_gemm_workspace_bytes(int64_t M, int64_t N, int64_t K) {
    if (M <= 0 || N <= 0 || !gemm_k_ok(K)) return CURVEFP_ERR_SHAPE;
    return gemm_workspace_bytes(M, N, K);
}

int curvefp_gemm_ws(const void* a_codes, const int8_t* a_scales, const void* b_codes, const int8_t* b_scales,
                    int64_t M, int64_t N, int64_t K, int format, int block, float* c, int64_t ldc,
                    void* workspace, int64_t workspace_bytes, void* stream) {
    if (!a_codes || !a_scales || !b_codes || !b_scales || !c || !workspace) return CURVEFP_ERR_NULL;
    if (!fmt_ok(format)) return CURVEFP_ERR_FORMAT;
    if (!block_ok(block)) return CURVEFP_ERR_BLOCK;
    if (M <= 0 || N <= 0 || !gemm_k_ok(K) || K % block || ldc < N) return CURVEFP_ERR_SHAPE;
    if (workspace_bytes < gemm_workspace_bytes(M, N, K)) return CURVEFP_ERR_SHAPE;
    if (!aligned16(a_codes) || !aligned16(b_codes) || !aligned16(c)) return CURVEFP_ERR_ALIGN;
    if (reinterpret_cast<uintptr_t>(workspace) % 256) return CURVEFP_ERR_ALIGN;
    return hip_status(launch_gemm_ws(a_codes, a_scales, b_codes, b_scales, M, N, K, format, block, c, ldc, workspace,
                                     reinterpret_cast<hipStream_t>(stream)));
}

int64_t curvefp_prepared_bytes(int64_t rows, int64_t k, int trans) {
    if (rows <= 0 || !gemm_k_ok(k) || (trans != 0 && trans != 1)) return CURVEFP_ERR_SHAPE;
    return prepared_bytes(rows, k, trans);
}

int curvefp_prepare(const void* codes, const int8_t* scales, int64_t rows, int64_t k, int format, int block,
                    int trans, void* prepared, int64_t prepared_size, void* stream) {
    if (!codes || !scales || !prepared) return CURVEFP_ERR_NULL;
    if (!fmt_ok(format)) return CURVEFP_ERR_FORMAT;
    if (!block_ok(block) || (trans != 0 && trans != 1)) return CURVEFP_ERR_BLOCK;
    if (rows <= 0 || !gemm_k_ok(k)) return CURVEFP_ERR_SHAPE;
    // blocks along k (trans 0) or along the rows of the reused operand (trans 1), whose expansion
    // grid has one workgroup row per 256 rows
    if (trans ? (rows % block || (rows + 255) / 256 > 65535) : k % block) return CURVEFP_ERR_SHAPE;
    if (prepared_size < prepared_bytes(rows, k, trans)) return CURVEFP_ERR_SHAPE;
    if (!aligned16(codes) || reinterpret_cast<uintptr_t>(prepared) % 256) return CURVEFP_ERR_ALIGN;
    return hip_status(launch_prepare(codes, scales, rows, k, format, block, trans, prepared,
                                     reinterpret_cast<hipStream_t>(stream)));
}

int curvefp_quantize_prepare(const void* src, int dtype, int64_t rows, int64_t k, int64_t ld_src, int format,
                             int block, void* codes, int8_t* scales, void* prepared, int64_t prepared_size, float* dst,
                             int64_t ld_dst, void* stream) {
    const int st = qp_check(dtype, k, format, block, src, rows, ld_src, codes, scales, prepared, prepared_size, dst,
                            ld_dst);
    if (st != CURVEFP_OK) return st;
    return hip_status(launch_quantize_prepare(src, dtype, rows, k, ld_src, format, block, codes, scales, prepared, dst,
                                              ld_dst, reinterpret_cast<hipStream_t>(stream)));
}

int curvefp_quantize_prepare_pair(const void* src_a, int64_t rows_a, int64_t ld_a, void* codes_a, int8_t* scales_a,
                                  void* prepared_a, int64_t prepared_a_size, float* dst_a, int64_t ld_dst_a,
                                  const void* src_b, int64_t rows_b, int64_t ld_b, void* codes_b, int8_t* scales_b,
                                  void* prepared_b, int64_t prepared_b_size, float* dst_b, int64_t ld_dst_b,
                                  int dtype, int64_t k, int format, int block, void* stream) {
    int st = qp_check(dtype, k, format, block, src_a, rows_a, ld_a, codes_a, scales_a, prepared_a, prepared_a_size,
                      dst_a, ld_dst_a);
    if (st != CURVEFP_OK) return st;
    st = qp_check(dtype, k, format, block, src_b, rows_b, ld_b, codes_b, scales_b, prepared_b, prepared_b_size, dst_b,
                  ld_dst_b);
    if (st != CURVEFP_OK) return st;
    if (rows_a + rows_b >= ((int64_t)1 << 31)) return CURVEFP_ERR_SHAPE;
    return hip_status(launch_quantize_prepare_pair(src_a, rows_a, ld_a, codes_a, scales_a, prepared_a, dst_a, ld_dst_a,
                                                   src_b, rows_b, ld_b, codes_b, scales_b, prepared_b, dst_b, ld_dst_b,
                                                   dtype, k, format, block, reinterpret_cast<hipStream_t>(stream)));
}

int64_t curvefp_gemm_prepared_workspace_bytes(int64_t M, int64_t N, int64_t K) {
    if (M <= 0 || N <= 0 || !gemm_k_ok(K)) return CURVEFP_ERR_SHAPE;
    return gemm_prepared_workspace_bytes(M, N, K);
}

int curvefp_gemm_prepared(const void* a_prepared, int format_a, const void* b_prepared, int format_b, int64_t M,
                          int64_t N, int64_t K, float* c, int64_t ldc, void* workspace, int64_t workspace_bytes,
                          void* stream) {
    if (!a_prepared || !b_prepared || !c) return CURVEFP_ERR_NULL;
    if (!fmt_ok(format_a) || !fmt_ok(format_b)) return CURVEFP_ERR_FORMAT;
    if (M <= 0 || N <= 0 || !gemm_k_ok(K) || ldc < N) return CURVEFP_ERR_SHAPE;
    const int64_t need = gemm_prepared_workspace_bytes(M, N, K);
    if (need > 0 && !workspace) return CURVEFP_ERR_NULL;
    if (workspace_bytes < need) return CURVEFP_ERR_SHAPE;
    if (reinterpret_cast<uintptr_t>(a_prepared) % 256 || reinterpret_cast<uintptr_t>(b_prepared) % 256 ||
        !aligned16(c) || reinterpret_cast<uintptr_t>(workspace) % 256)
        return CURVEFP_ERR_ALIGN;
    return hip_status(launch_gemm_prepared(a_prepared, format_a, b_prepared, format_b, M, N, K, c, ldc, workspace,
                                           reinterpret_cast<hipStream_t>(stream)));
}

int curvefp_gemm_ws_static(const void* a_codes, const int8_t* a_scales, const void* b_codes,
                           const int8_t* b_scales, int64_t M, int64_t N, int64_t K, int format, int block, float* c,
                           int64_t ldc, void* stream) {
    if (!a_codes || !a_scales || !b_codes || !b_scales || !c) return CURVEFP_ERR_NULL;
    if (!fmt_ok(format)) return CURVEFP_ERR_FORMAT;
    if (!block_ok(block)) return CURVEFP_ERR_BLOCK;
    if (M <= 0 || N <= 0 || !gemm_k_ok(K) || K % block || ldc < N) return CURVEFP_ERR_SHAPE;
    if (gemm_workspace_bytes(M, N, K) > CURVEFP_STATIC_SCRATCH_BYTES) return CURVEFP_ERR_SHAPE;
    if (!aligned16(a_codes) || !aligned16(b_codes) || !aligned16(c)) return CURVEFP_ERR_ALIGN;
    void* ws = nullptr;
    if (static_scratch(&ws) != hipSuccess) return CURVEFP_ERR_HIP;
    return hip_status(launch_gemm_ws(a_codes, a_scales, b_codes, b_scales, M, N, K, format, block, c, ldc, ws,
                                     reinterpret_cast<hipStream_t>(stream)));
}

int curvefp_gemm_requant(const void* a_codes, const int8_t* a_scales, const void* b_codes, const int8_t* b_scales,
                         int64_t M, int64_t N, int64_t K, int format, int block, int out_format, int out_block,
                         void* out_codes, int8_t* out_scales, void* workspace, int64_t workspace_bytes,
                         void* stream) {
    if (!a_codes || !a_scales || !b_codes || !b_scales || !out_codes || !out_scales || !workspace)
        return CURVEFP_ERR_NULL;
    if (!fmt_ok(format) || !fmt_ok(out_format)) return CURVEFP_ERR_FORMAT;
    if (!block_ok(block)) return CURVEFP_ERR_BLOCK;
    // output blocks lie inside one 256-column tile of the epilogue
    if (out_block != 32 && out_block != 64 && out_block != 128 && out_block != 256) return CURVEFP_ERR_BLOCK;
    if (M <= 0 || N <= 0 || !gemm_k_ok(K) || K % block || N % out_block) return CURVEFP_ERR_SHAPE;
    if (workspace_bytes < gemm_workspace_bytes(M, N, K)) return CURVEFP_ERR_SHAPE;
    if (!aligned16(a_codes) || !aligned16(b_codes) || !aligned16(out_codes)) return CURVEFP_ERR_ALIGN;
    if (reinterpret_cast<uintptr_t>(workspace) % 256) return CURVEFP_ERR_ALIGN;
    return hip_status(launch_gemm_requant(a_codes, a_scales, b_codes, b_scales, M, N, K, format, block, out_format,
                                          out_block, out_codes, out_scales, workspace,
                                          reinterpret_cast<hipStream_t>(stream)));
}

int64_t curvefp_gemm_mixed_workspace_bytes(int64_t M, int64_t N, int64_t K) {
    if (M <= 0 || N <= 0 || !gemm_k_ok(K)) return CURVEFP_ERR_SHAPE;
    return gemm_mixed_workspace_bytes(M, N, K);
}

int curvefp_gemm_mixed(const void* a_codes, const int8_t* a_scales, int a_format, int a_trans,
                       const void* b_codes, const int8_t* b_scales, int b_format, int b_trans,
                       int64_t M, int64_t N, int64_t K, int block, float* c, int64_t ldc,
                       void* workspace, int64_t workspace_bytes, void* stream) {
    if (!a_codes || !a_scales || !b_codes || !b_scales || !c || !workspace) return CURVEFP_ERR_NULL;
    if (!fmt_ok(a_format) || !fmt_ok(b_format)) return CURVEFP_ERR_FORMAT;
    if (!block_ok(block) || (a_trans != 0 && a_trans != 1) || (b_trans != 0 && b_trans != 1)) return CURVEFP_ERR_BLOCK;
    if (M <= 0 || N <= 0 || !gemm_k_ok(K) || ldc < N) return CURVEFP_ERR_SHAPE;
    // an operand quantized along K has its blocks along K; a reused operand has them along its
    // GEMM rows; the expansion grid has one workgroup row per 256 GEMM rows of each reused
    // operand (at most 65535 in all)
    if ((!a_trans || !b_trans) && K % block) return CURVEFP_ERR_SHAPE;
    if ((a_trans && M % block) || (b_trans && N % block)) return CURVEFP_ERR_SHAPE;
    if ((a_trans ? (M + 255) / 256 : 0) + (b_trans ? (N + 255) / 256 : 0) > 65535) return CURVEFP_ERR_SHAPE;
    if (workspace_bytes < gemm_mixed_workspace_bytes(M, N, K)) return CURVEFP_ERR_SHAPE;
    if (!aligned16(a_codes) || !aligned16(b_codes) || !aligned16(c)) return CURVEFP_ERR_ALIGN;
    if (reinterpret_cast<uintptr_t>(workspace) % 256) return CURVEFP_ERR_ALIGN;
    return hip_status(launch_gemm_mixed(a_codes, a_scales, a_format, a_trans, b_codes, b_scales, b_format, b_trans,
                                        M, N, K, block, c, ldc, workspace, reinterpret_cast<hipStream_t>(stream)));
}

const char* curvefp_status_string(int status) {
    switch (status) {
        case CURVEFP_OK: return "ok";
        case CURVEFP_ERR_NULL: return "null pointer argument";
        case CURVEFP_ERR_SHAPE:
            return "invalid shape, leading dimension, count, or blocked extent not a multiple of the block";
        case CURVEFP_ERR_FORMAT: return "unknown format or dtype";
        case CURVEFP_ERR_BLOCK: return "unsupported block size, block axis or scale width";
        case CURVEFP_ERR_ALIGN: return "pointer or row not 16-byte aligned";
        case CURVEFP_ERR_HIP: return "HIP error (kernel launch)";
        default: return "unknown status";
    }
}

}  // extern "C"
#pragma GCC visibility pop
