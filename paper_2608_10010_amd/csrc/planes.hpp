// Expanded GEMM operands ("planes"): the layout and arithmetic shared by the GEMM's own expansion
// kernels and by the fused quantize-and-prepare kernel, which must write the same bytes.
//
// An operand with R rows over K is stored per K block of 32 and per tile of 256 rows as two
// 16 KB planes, hi then lo: fp16 pairs with hi + lo = 2^{x} 2^{f/N} to 22 significant bits for
// every code (the level r^{n/K} = 2^{w + f/N} of Eq. curvefp-value), where x = (a_b - alpha) +
// w + bias carries the code's block scale a_b relative to alpha, the largest block scale of its
// row.  A tile row is 64 bytes (32 halves) with its four 16-byte chunks XOR-swizzled so that the
// GEMM's fragment reads spread over the LDS banks.
#pragma once

#include <cstdint>
#include <hip/hip_runtime.h>

namespace curvefp {

typedef _Float16 half2v __attribute__((ext_vector_type(2)));

constexpr int BM = 256, BK = 32;
constexpr int ROW_BYTES = BK * 2;                 // one fp16 plane row: 32 halves
constexpr int PLANE = BM * ROW_BYTES;             // 16 KB: one hi or lo plane of a 256-row tile

// Row maxima of block scales are taken over keys: a block that held a NaN or an infinity (scale
// -128) counts as POISON_KEY, above every scale, so a row's maximum is at least POISON_KEY exactly
// when one of its blocks is poisoned.  Such a row's expansion then flushes every element (its
// offsets to the maximum are hundreds of binades), and the GEMM's epilogue writes NaN for each
// output in that row or column.
constexpr int POISON_KEY = 0x4000;
__device__ __forceinline__ int scale_key(int s) { return s == -128 ? POISON_KEY : s; }

// byte offset of 16-byte chunk q (k = 8q .. 8q+7) of tile row r
__device__ __forceinline__ int swz(int r, int q) { return r * ROW_BYTES + 16 * (q ^ (((r >> 1) ^ (r >> 3)) & 3)); }

__device__ __forceinline__ uint32_t f16_pow2_neg(int d) {
    // bits of the fp16 value 2^-d for 0 <= d <= 24 (exact: subnormal below 2^-14)
    const _Float16 m = __builtin_amdgcn_ldexph((_Float16)1.0f, -d);
    return (uint32_t)__builtin_bit_cast(uint16_t, m);
}

__device__ __forceinline__ uint32_t pk_mul(uint32_t x, half2v m) {
    return __builtin_bit_cast(uint32_t, __builtin_bit_cast(half2v, x) * m);
}

// one 16-byte chunk of both planes: e[i] = the expansion table's entry (lo16 << 16 | hi16) of
// code i at its row's largest scale, D = alpha - a_b >= 0 the block's offset below it; each pair
// is scaled by 2^-min(D, 24), and by 2^-min(D - 24, 24) more when D > 24 (exact while the result
// stays normal, correctly rounded below)
__device__ __forceinline__ void expand_chunk8(const uint32_t* e, int D, uint32_t* hv, uint32_t* lv) {
    const half2v m1 = __builtin_bit_cast(half2v, f16_pow2_neg(min(max(D, 0), 24)) * 0x10001u);
#pragma unroll
    for (int p = 0; p < 4; p++) {
        hv[p] = pk_mul(__builtin_amdgcn_perm(e[2 * p + 1], e[2 * p], 0x05040100u), m1);
        lv[p] = pk_mul(__builtin_amdgcn_perm(e[2 * p + 1], e[2 * p], 0x07060302u), m1);
    }
    if (D > 24) {   // a block more than 24 binades below its row's top: second multiply
        const half2v m2 = __builtin_bit_cast(half2v, f16_pow2_neg(min(D - 24, 24)) * 0x10001u);
#pragma unroll
        for (int p = 0; p < 4; p++) {
            hv[p] = pk_mul(hv[p], m2);
            lv[p] = pk_mul(lv[p], m2);
        }
    }
}

}  // namespace curvefp
