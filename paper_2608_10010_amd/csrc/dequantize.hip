// CurveFP reconstruction x_hat = (-1)^s 2^{a_b} r^{e + k/K} (Eq. curvefp-value),
// written as the nearest fp32 value.  With r = 2^{P/Q} the magnitude is 2^{w + f/N},
// w = floor(P n / N), f = P n mod N, N = QK (binary radix: w = e, f = k).
//
// In the normal range the result is exact bit assembly: the fp32 exponent is
// w + a_b and the mantissa is that of fl32(2^{f/N}) (scaling by a power of two
// commutes with rounding there).  Below 2^-126 the 62-bit significand of
// 2^{f/N} is rounded once at the subnormal position.  HBM-bound: one byte (or 7
// bits) and 1/32 scale byte read, four bytes written per element.
#include "curvefp_internal.hpp"
#include "codec.hpp"
#include "device_util.hpp"
#include "curvefp_tables.inc"

#include <cstring>

namespace curvefp {

// compile-time tables (curvefp_tables.inc, written at build time by gen_tables)
__constant__ uint32_t g_mant[NUM_FORMATS][8] = CURVEFP_MANT_INIT;
__constant__ uint64_t g_sig62[NUM_FORMATS][8] = CURVEFP_SIG62_INIT;
// rational radix: per magnitude rank, (w << 24) | mantissa of fl32(2^{f/N}) and floor(2^{f/N} 2^62)
__constant__ uint32_t g_dq_em[NUM_FORMATS][128] = CURVEFP_DQ_EM_INIT;
__constant__ uint64_t g_dq_sig62[NUM_FORMATS][128] = CURVEFP_DQ_SIG62_INIT;

namespace {

// chunk g = 8 consecutive codes: chunk g mod cpr of row g / cpr, block g / 4 (blocks are
// contiguous in the code and scale arrays); a grid-stride loop over the chunks, one per thread
// per round (a capped grid with plain stores measured fastest for this write-heavy stream; the
// cap grows with the tensor, see the launch), or with TWO, two rounds per pass whose loads are
// all issued before the first chunk is written
template <class F, bool TWO>
__global__ __launch_bounds__(256) void dequantize_kernel(
    const uint8_t* __restrict__ codes, const int8_t* __restrict__ scales, uint32_t nchunks, uint32_t cpr,
    Div32 dcpr, int64_t ld, float* __restrict__ dst, int fidx, Div32 dgq) {
    constexpr int TAB = F::BINARY ? 8 : 128;
    __shared__ uint32_t mant[TAB];
    __shared__ uint64_t sig[TAB];
    if (threadIdx.x < TAB) {
        mant[threadIdx.x] = F::BINARY ? g_mant[fidx][threadIdx.x] : g_dq_em[fidx][threadIdx.x];
        sig[threadIdx.x] = F::BINARY ? g_sig62[fidx][threadIdx.x] : g_dq_sig62[fidx][threadIdx.x];
    }
    __syncthreads();
    const bool dense = ld == (int64_t)cpr * 8;
    const uint32_t stride = gridDim.x * 256u;
    // the words of chunk g (8 codes) and its block's scale
    auto fetch = [&](uint32_t g, uint2& w, uint32_t& w2, int& a) {
        const uint32_t b = g >> 2;                  // 32-element group; its scale is that of block b / (G / 32)
        a = scales[div32(b, dgq)];
        if (!F::PACKED7) {
            w = *reinterpret_cast<const uint2*>(codes + (uint64_t)g * 8);
            w2 = 0u;
        } else {
            // bytes [7 part, 7 part + 7) of the block's 28 bytes; parts 1 and 2 (bytes 7..13 and
            // 14..20) straddle three dwords, parts 0 and 3 two
            const uint32_t* base = reinterpret_cast<const uint32_t*>(codes + (uint64_t)b * 28);
            const int part = (int)(g & 3);
            const int d0 = (7 * part) >> 2;
            w = make_uint2(base[d0], base[d0 + 1]);
            w2 = (part == 1 || part == 2) ? base[d0 + 2] : 0u;
        }
    };
    auto emit = [&](uint32_t g, uint2 w, uint32_t w2, int a) {
        uint32_t c[8];
        if (!F::PACKED7) {
#pragma unroll
            for (int i = 0; i < 4; i++) {
                c[i] = (w.x >> (8 * i)) & 0xFFu;
                c[4 + i] = (w.y >> (8 * i)) & 0xFFu;
            }
        } else {
            const int part = (int)(g & 3);
            const int off = 7 * part - 4 * ((7 * part) >> 2);
            const uint64_t lo = (uint64_t)w.x | ((uint64_t)w.y << 32);
            const uint64_t hi = w2;
            const uint64_t chunk = off ? ((lo >> (8 * off)) | (hi << (64 - 8 * off))) : lo;
#pragma unroll
            for (int i = 0; i < 8; i++) c[i] = (uint32_t)(chunk >> (7 * i)) & 0x7Fu;
        }
        uint32_t o[8];
        if (a == -128) {
#pragma unroll
            for (int i = 0; i < 8; i++) o[i] = 0x7FC00000u;   // poisoned block
        } else {
#pragma unroll
            for (int i = 0; i < 8; i++) o[i] = value_bits<F>(c[i], a, mant, sig);
        }
        int64_t e;
        if (dense) {
            e = (int64_t)g * 8;
        } else {
            const uint32_t r = div32(g, dcpr);
            e = (int64_t)r * ld + (int64_t)(g - r * cpr) * 8;
        }
        uint4* out = reinterpret_cast<uint4*>(dst + e);
        out[0] = make_uint4(o[0], o[1], o[2], o[3]);
        out[1] = make_uint4(o[4], o[5], o[6], o[7]);
    };
    if (!TWO) {
        for (uint32_t g = blockIdx.x * 256u + threadIdx.x; g < nchunks; g += stride) {
            uint2 w;
            uint32_t x;
            int a;
            fetch(g, w, x, a);
            emit(g, w, x, a);
        }
        return;
    }
    // large grids: two chunks per thread and pass (g and g + stride), both requested before either
    // is written (64-bit positions: g + 2 stride can pass 2^32)
    for (uint64_t p = (uint64_t)blockIdx.x * 256u + threadIdx.x; p < nchunks; p += 2ull * stride) {
        const uint32_t g0 = (uint32_t)p;
        const bool two = p + stride < nchunks;
        const uint32_t g1 = two ? (uint32_t)(p + stride) : g0;
        uint2 w0, w1 = make_uint2(0u, 0u);
        uint32_t x0, x1 = 0u;
        int a0, a1 = 0;
        fetch(g0, w0, x0, a0);
        if (two) fetch(g1, w1, x1, a1);
        emit(g0, w0, x0, a0);
        if (two) emit(g1, w1, x1, a1);
    }
}

template <class F>
hipError_t launch_fmt(const void* codes, const int8_t* scales, int64_t outer, int64_t k, int block, float* dst,
                      int64_t ld, int fidx, hipStream_t s) {
    const Div32 dgq = make_div32((uint32_t)(block / 32));
    const int64_t cpr = k / 8;
    const int64_t slab = ((int64_t)1 << 31) / cpr;   // 32-bit chunk indices per launch
    const uint8_t* cp = reinterpret_cast<const uint8_t*>(codes);
    for (int64_t r0 = 0; r0 < outer; r0 += slab) {
        const int64_t nr = outer - r0 < slab ? outer - r0 : slab;
        const int64_t nchunks = nr * cpr;
        // two chunks per thread (two rounds) once that takes more than 8192 workgroups, else at
        // most 8192: on 8192 x 4096 codes more workgroups measured slower, on 32768 x 8192 the
        // 8192 cap 13% slower than two rounds
        const int64_t half = (nchunks + 511) / 512;
        int64_t blocks = (nchunks + 255) / 256;
        const int64_t cap = half > 8192 ? half : 8192;
        blocks = blocks < cap ? blocks : cap;
        // the two rounds of large grids with both chunks' loads in flight at once (16% faster on
        // 32768 x 8192 from HBM; on grids of at most 8192 workgroups the plain loop measured faster)
        const uint8_t* cr = cp + (F::PACKED7 ? r0 * (k / 32) * 28 : r0 * k);
        if (half > 8192)
            hipLaunchKernelGGL((dequantize_kernel<F, true>), dim3((unsigned)blocks), dim3(256), 0, s, cr,
                               scales + r0 * (k / block), (uint32_t)nchunks, (uint32_t)cpr,
                               make_div32((uint32_t)cpr), ld, dst + r0 * ld, fidx, dgq);
        else
            hipLaunchKernelGGL((dequantize_kernel<F, false>), dim3((unsigned)blocks), dim3(256), 0, s, cr,
                               scales + r0 * (k / block), (uint32_t)nchunks, (uint32_t)cpr,
                               make_div32((uint32_t)cpr), ld, dst + r0 * ld, fidx, dgq);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace

hipError_t launch_dequantize(const void* codes, const int8_t* scales, int format, int64_t outer,
                             int64_t k, int block, float* dst, int64_t ld_dst, hipStream_t s) {
    switch (format) {
        case 0: return launch_fmt<FmtE4C3>(codes, scales, outer, k, block, dst, ld_dst, 0, s);
        case 1: return launch_fmt<FmtE5C2>(codes, scales, outer, k, block, dst, ld_dst, 1, s);
        case 2: return launch_fmt<FmtE3C3>(codes, scales, outer, k, block, dst, ld_dst, 2, s);
        case 3: return launch_fmt<FmtE4C3R89>(codes, scales, outer, k, block, dst, ld_dst, 3, s);
        default: return launch_fmt<FmtE4C3R34>(codes, scales, outer, k, block, dst, ld_dst, 4, s);
    }
}

}  // namespace curvefp
