// Element arithmetic shared by several kernels: the CurveFP reconstruction x_hat =
// (-1)^s 2^{a_b} r^{e + k/K} (Eq. curvefp-value) as fp32 bits (dequantize kernel, static-scale
// quantizer), and the block quantizer's rule with the format's constants given at run time
// (the GEMM's output requantization).
#pragma once

#include <cstdint>
#include <hip/hip_runtime.h>

#include "curvefp_internal.hpp"

namespace curvefp {

// binary radix: mant/sig indexed by the curve index k (8 entries); rational radix: by the
// magnitude rank (128 entries, mant holding (w << 24) | mantissa)
template <class F>
__device__ __forceinline__ uint32_t value_bits(uint32_t code, int a, const uint32_t* mant, const uint64_t* sig) {
    const uint32_t m = code & F::MAG_MASK;
    if (m == 0) return 0u;
    const uint32_t s = (code >> F::EC) & 1u;
    int ex, k;
    uint32_t mbits;
    if (F::BINARY) {
        const int n = (int)m - F::B;
        k = n & (F::K - 1);
        ex = (n >> F::C) + a;                // floor(n / K) + a
        mbits = mant[k];
    } else {
        k = (int)m;
        const uint32_t em = mant[m];
        ex = ((int32_t)em >> 24) + a;        // floor(P n / N) + a
        mbits = em & 0x7FFFFFu;
    }
    uint32_t bits;
    if (ex > 127) {
        bits = 0x7F800000u;                  // beyond FLT_MAX: rounds to infinity
    } else if (ex >= -126) {
        bits = ((uint32_t)(ex + 127) << 23) | mbits;
    } else {
        const int sh = -87 - ex;             // 62 - (ex + 149), in [40, 56]
        const uint64_t v = sig[k];
        uint64_t q = v >> sh;
        const uint64_t rem = v & ((1ull << sh) - 1);
        const uint64_t half = 1ull << (sh - 1);
        q += (rem > half || (rem == half && (q & 1))) ? 1 : 0;
        bits = (uint32_t)q;
    }
    return bits | (s << 31);
}

// The quantizer of Sec. 3.1 with run-time format constants: the same decisions as the quantize
// kernels (quantize.hip: block_scale, scale_of, rank_exact, rank_lookup), for kernels that
// quantize values they have computed themselves.
struct QRule {
    int oz;               // octave of the zero threshold (first table octave)
    int ohi;              // octave of the top level
    int qsize;            // table entries, (ohi - oz + 1) * 128
    int ec;               // E + C: the sign bit's position
    uint32_t lmax_mant;   // mantissa field of fl32 of the top level
};

// ceil-absmax block scale from the largest magnitude's fp32 bits: -128 for a non-finite block
__device__ __forceinline__ int qr_scale(uint32_t amax, const QRule& q) {
    if (amax >= 0x7F800000u) return -128;
    const int ef = (int)(amax >> 23);
    if (ef == 0) return -127;                        // all zero, or a subnormal maximum
    const int a = ef - 127 - q.ohi + (((amax & 0x7FFFFFu) > q.lmax_mant) ? 1 : 0);
    return min(max(a, -127), 127);
}

// The rank of |x| (fp32 bits without the sign) at scale a in three steps, so that a caller can
// make all its table lookups at once: the scaled magnitude's bits (subnormal inputs normalized
// first), the table index, and the rank from the table entry (0 for zero, a poisoned scale, or a
// magnitude below the table).  Branch-free.
__device__ __forceinline__ int32_t qr_scaled(uint32_t mag, int a) {
    const int p = 31 - __clz(mag | 1u);              // leading one of a subnormal input
    const uint32_t mn = mag << max(23 - p, 0);
    const int32_t ysub = (int32_t)(((uint32_t)(p - 22 - a) << 23) | (mn & 0x7FFFFFu));
    return (mag >> 23) == 0 ? ysub : (int32_t)mag - (a << 23);
}

__device__ __forceinline__ int32_t qr_index(int32_t yb, const QRule& q) { return (yb >> 16) - ((127 + q.oz) << 7); }

__device__ __forceinline__ uint32_t qr_from_entry(uint32_t e, int32_t yb, int32_t idx, uint32_t mag, int a) {
    const uint32_t r = (e >> 16) + ((((uint32_t)yb & 0xFFFFu) > (e & 0xFFFFu)) ? 1u : 0u);
    return (idx < 0 || mag == 0 || a == -128) ? 0u : r;
}

// magnitude rank of |x| at scale a, lut = the format's table
__device__ __forceinline__ uint32_t qr_rank(uint32_t mag, int a, const uint32_t* lut, const QRule& q) {
    const int32_t yb = qr_scaled(mag, a);
    const int32_t idx = qr_index(yb, q);
    return qr_from_entry(lut[min(max(idx, 0), q.qsize - 1)], yb, idx, mag, a);
}

}  // namespace curvefp
