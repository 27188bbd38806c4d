// The CurveFP reconstruction x_hat = (-1)^s 2^{a_b} r^{e + k/K} (Eq. curvefp-value) as fp32 bits,
// shared by the dequantize kernel and the static-scale (MSE) quantizer.
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

}  // namespace curvefp
