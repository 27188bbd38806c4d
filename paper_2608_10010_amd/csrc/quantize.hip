// CurveFP block quantization Q(X) on gfx950 (Sec. 3.1 of the CurveFP paper).
//
// For a block of 32 values with maximum magnitude amax:
//   scale  a = smallest integer with amax <= 2^a * fl32(2^{n_max/K})  (ceil-absmax),
//          computed on the fp32 bit pattern: a = e(amax) - o_hi + [mant(amax) > mant(fl32(L_max))];
//   element: y = |x| 2^{-a} is formed exactly by subtracting a from the exponent
//          field; its rank is looked up in a per-format table indexed by the
//          bfloat16-truncated bits of y over the octaves that can reach a nonzero
//          code, plus one compare of the low 16 bits against the single decision
//          point a table bucket can hold.  The table encodes the nearest-level rule
//          (nearest in absolute error, saturating at the endpoints) derived on the host.
// Memory: HBM-bound; one pass, coalesced 16-byte loads, one byte (or 7 bits)
// per code and one byte per block written.
#include "curvefp_internal.hpp"
#include "device_util.hpp"

#include <cstring>

namespace curvefp {

__device__ uint32_t g_qlut[3][QLUT_MAX];
__device__ uint32_t g_lmax_mant[3];

hipError_t quantize_upload(const AllTables& t) {
    static uint32_t h[3][QLUT_MAX];
    uint32_t lm[3];
    for (int f = 0; f < 3; f++) {
        memcpy(h[f], t.f[f].qlut, sizeof(h[f]));
        lm[f] = t.f[f].lmax_mant;
    }
    hipError_t e = hipMemcpyToSymbol(HIP_SYMBOL(g_qlut), h, sizeof(h));
    if (e != hipSuccess) return e;
    return hipMemcpyToSymbol(HIP_SYMBOL(g_lmax_mant), lm, sizeof(lm));
}

namespace {

template <class F>
__device__ __forceinline__ int block_scale(uint32_t amax, uint32_t lmax_mant) {
    if (amax == 0) return 0;
    const int ef = (int)(amax >> 23);
    if (ef == 0) return -127;                       // subnormal maximum: below every clamp
    const int a = ef - 127 - F::OHI + (((amax & 0x7FFFFFu) > lmax_mant) ? 1 : 0);
    return min(max(a, -127), 127);
}

// rank of y whose fp32 bit pattern is yb (already scaled), table in LDS
template <class F>
__device__ __forceinline__ uint32_t rank_lookup(int32_t yb, const uint32_t* lut) {
    int32_t idx = (yb >> 16) - ((127 + F::OZ) << 7);
    if (idx < 0) return 0;
    idx = min(idx, F::QLUT_SIZE - 1);
    const uint32_t e = lut[idx];
    return (e >> 16) + ((((uint32_t)yb & 0xFFFFu) > (e & 0xFFFFu)) ? 1u : 0u);
}

// fast path: a >= A_FAST_MIN, where subnormal or zero inputs can only reach rank 0
template <class F>
__device__ __forceinline__ uint32_t rank_fast(uint32_t mag, int a, const uint32_t* lut) {
    return rank_lookup<F>((int32_t)mag - (a << 23), lut);
}

// exact path for blocks with tiny scales: normalize subnormal inputs first
template <class F>
__device__ __forceinline__ uint32_t rank_exact(uint32_t mag, int a, const uint32_t* lut) {
    if (mag == 0) return 0;
    int32_t yb;
    if ((mag >> 23) == 0) {
        const int p = 31 - __clz(mag);              // position of the leading one, 0..22
        const uint32_t mn = mag << (23 - p);
        yb = (int32_t)(((uint32_t)(p - 22 - a) << 23) | (mn & 0x7FFFFFu));
    } else {
        yb = (int32_t)mag - (a << 23);
    }
    return rank_lookup<F>(yb, lut);
}

template <class F>
__device__ __forceinline__ void ranks_of(const uint32_t* mag, int n, int a, const uint32_t* lut,
                                         uint32_t* r) {
    if (a == -128) {
        for (int i = 0; i < n; i++) r[i] = 0;
    } else if (a >= F::A_FAST_MIN) {
        for (int i = 0; i < n; i++) r[i] = rank_fast<F>(mag[i], a, lut);
    } else {
        for (int i = 0; i < n; i++) r[i] = rank_exact<F>(mag[i], a, lut);
    }
}

template <class F>
__device__ __forceinline__ int scale_of(uint32_t amax, uint32_t lmax_mant) {
    return (amax >= 0x7F800000u) ? -128 : block_scale<F>(amax, lmax_mant);
}

template <bool BF16>
__device__ __forceinline__ void load8(const void* src, int64_t elem, uint32_t* mag, uint32_t* sgn) {
    if (BF16) {
        const uint4 v = *reinterpret_cast<const uint4*>(reinterpret_cast<const uint16_t*>(src) + elem);
        const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int i = 0; i < 4; i++) {
            mag[2 * i] = (w[i] << 16) & 0x7FFF0000u;
            mag[2 * i + 1] = w[i] & 0x7FFF0000u;
            sgn[2 * i] = (w[i] >> 15) & 1u;
            sgn[2 * i + 1] = w[i] >> 31;
        }
    } else {
        const uint4* p = reinterpret_cast<const uint4*>(reinterpret_cast<const uint32_t*>(src) + elem);
        const uint4 v0 = p[0], v1 = p[1];
        const uint32_t w[8] = {v0.x, v0.y, v0.z, v0.w, v1.x, v1.y, v1.z, v1.w};
#pragma unroll
        for (int i = 0; i < 8; i++) {
            mag[i] = w[i] & 0x7FFFFFFFu;
            sgn[i] = w[i] >> 31;
        }
    }
}

// 4 threads per block of 32 along a row; each thread owns 8 consecutive elements
template <class F, bool BF16>
__global__ __launch_bounds__(256) void quantize_rows_kernel(
    const void* __restrict__ src, int64_t rows, int64_t cols, int64_t ld,
    uint8_t* __restrict__ codes, int8_t* __restrict__ scales, int fidx) {
    __shared__ uint32_t lut[F::QLUT_SIZE];
    for (int i = threadIdx.x; i < F::QLUT_SIZE; i += blockDim.x) lut[i] = g_qlut[fidx][i];
    const uint32_t lmax_mant = g_lmax_mant[fidx];
    __syncthreads();

    const int64_t bpr = cols / 32;
    const int64_t nthreads = rows * bpr * 4;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; g < nthreads; g += stride) {
        const int64_t b = g >> 2;
        const int part = (int)(g & 3);
        const int64_t r = b / bpr;
        const int64_t cb = b - r * bpr;
        uint32_t mag[8], sgn[8];
        load8<BF16>(src, r * ld + cb * 32 + part * 8, mag, sgn);
        uint32_t amax = 0;
#pragma unroll
        for (int i = 0; i < 8; i++) amax = max(amax, mag[i]);
        amax = quad_max_u32(amax);
        const int a = scale_of<F>(amax, lmax_mant);
        uint32_t rk[8];
        ranks_of<F>(mag, 8, a, lut, rk);
        uint32_t c[8];
#pragma unroll
        for (int i = 0; i < 8; i++) c[i] = rk[i] | ((rk[i] != 0 ? sgn[i] : 0u) << F::EC);
        if (!F::PACKED7) {
            uint2 o;
            o.x = c[0] | (c[1] << 8) | (c[2] << 16) | (c[3] << 24);
            o.y = c[4] | (c[5] << 8) | (c[6] << 16) | (c[7] << 24);
            *reinterpret_cast<uint2*>(codes + r * cols + cb * 32 + part * 8) = o;
        } else {
            // 56-bit chunk of this thread; the block string is chunk0 | chunk1 << 56 | ...
            uint64_t chunk = 0;
#pragma unroll
            for (int i = 0; i < 8; i++) chunk |= (uint64_t)c[i] << (7 * i);
            const uint32_t nlo = dpp_u32<QP_NEXT>((uint32_t)chunk);
            const uint32_t nhi = dpp_u32<QP_NEXT>((uint32_t)(chunk >> 32));
            const uint64_t next = ((uint64_t)nhi << 32) | nlo;
            uint32_t* base = reinterpret_cast<uint32_t*>(codes + (r * bpr + cb) * 28);
            if (part < 3) {
                const uint64_t lo64 = chunk | (next << 56);
                const uint64_t hi64 = next >> 8;
                const int sh = 8 * part;
                const uint64_t w = sh ? ((lo64 >> sh) | (hi64 << (64 - sh))) : lo64;
                base[2 * part] = (uint32_t)w;
                base[2 * part + 1] = (uint32_t)(w >> 32);
            } else {
                base[6] = (uint32_t)(chunk >> 24);
            }
        }
        if (part == 0) scales[r * bpr + cb] = (int8_t)a;
    }
}

// quantize-transpose: one thread per (column, block of 32 rows)
template <class F, bool BF16>
__global__ __launch_bounds__(256) void quantize_cols_kernel(
    const void* __restrict__ src, int64_t rows, int64_t cols, int64_t ld,
    uint8_t* __restrict__ codes, int8_t* __restrict__ scales, int fidx) {
    __shared__ uint32_t lut[F::QLUT_SIZE];
    for (int i = threadIdx.x; i < F::QLUT_SIZE; i += blockDim.x) lut[i] = g_qlut[fidx][i];
    const uint32_t lmax_mant = g_lmax_mant[fidx];
    __syncthreads();

    const int64_t rblocks = rows / 32;
    const int64_t total = rblocks * cols;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; g < total; g += stride) {
        const int64_t rb = g / cols;
        const int64_t c = g - rb * cols;
        uint32_t mag[32], sgn[32];
#pragma unroll
        for (int i = 0; i < 32; i++) {
            const int64_t e = (rb * 32 + i) * ld + c;
            uint32_t w = BF16 ? ((uint32_t)reinterpret_cast<const uint16_t*>(src)[e] << 16)
                              : reinterpret_cast<const uint32_t*>(src)[e];
            mag[i] = w & 0x7FFFFFFFu;
            sgn[i] = w >> 31;
        }
        uint32_t amax = 0;
#pragma unroll
        for (int i = 0; i < 32; i++) amax = max(amax, mag[i]);
        const int a = scale_of<F>(amax, lmax_mant);
        uint32_t rk[32];
        ranks_of<F>(mag, 32, a, lut, rk);
        uint32_t cc[32];
#pragma unroll
        for (int i = 0; i < 32; i++) cc[i] = rk[i] | ((rk[i] != 0 ? sgn[i] : 0u) << F::EC);
        if (!F::PACKED7) {
            uint4* o = reinterpret_cast<uint4*>(codes + c * rows + rb * 32);
#pragma unroll
            for (int q = 0; q < 2; q++) {
                uint4 v;
                v.x = cc[16 * q + 0] | (cc[16 * q + 1] << 8) | (cc[16 * q + 2] << 16) | (cc[16 * q + 3] << 24);
                v.y = cc[16 * q + 4] | (cc[16 * q + 5] << 8) | (cc[16 * q + 6] << 16) | (cc[16 * q + 7] << 24);
                v.z = cc[16 * q + 8] | (cc[16 * q + 9] << 8) | (cc[16 * q + 10] << 16) | (cc[16 * q + 11] << 24);
                v.w = cc[16 * q + 12] | (cc[16 * q + 13] << 8) | (cc[16 * q + 14] << 16) | (cc[16 * q + 15] << 24);
                o[q] = v;
            }
        } else {
            uint32_t w[7] = {0, 0, 0, 0, 0, 0, 0};
#pragma unroll
            for (int i = 0; i < 32; i++) {
                const int bit = 7 * i, d = bit >> 5, s = bit & 31;
                w[d] |= cc[i] << s;
                if (s > 25) w[d + 1] |= cc[i] >> (32 - s);
            }
            uint32_t* o = reinterpret_cast<uint32_t*>(codes + (c * rblocks + rb) * 28);
#pragma unroll
            for (int d = 0; d < 7; d++) o[d] = w[d];
        }
        scales[c * rblocks + rb] = (int8_t)a;
    }
}

template <class F>
hipError_t launch_fmt(const void* src, int dtype, int64_t rows, int64_t cols, int64_t ld, int axis,
                      int fidx, void* codes, int8_t* scales, hipStream_t s) {
    const int threads = 256;
    const int64_t work = axis == 1 ? rows * (cols / 32) * 4 : (rows / 32) * cols;
    int64_t blocks = (work + threads - 1) / threads;
    blocks = blocks < 8192 ? blocks : 8192;
    if (blocks < 1) blocks = 1;
    uint8_t* cp = reinterpret_cast<uint8_t*>(codes);
    if (axis == 1) {
        if (dtype == 1)
            hipLaunchKernelGGL((quantize_rows_kernel<F, true>), dim3(blocks), dim3(threads), 0, s, src, rows, cols, ld, cp, scales, fidx);
        else
            hipLaunchKernelGGL((quantize_rows_kernel<F, false>), dim3(blocks), dim3(threads), 0, s, src, rows, cols, ld, cp, scales, fidx);
    } else {
        if (dtype == 1)
            hipLaunchKernelGGL((quantize_cols_kernel<F, true>), dim3(blocks), dim3(threads), 0, s, src, rows, cols, ld, cp, scales, fidx);
        else
            hipLaunchKernelGGL((quantize_cols_kernel<F, false>), dim3(blocks), dim3(threads), 0, s, src, rows, cols, ld, cp, scales, fidx);
    }
    return hipGetLastError();
}

}  // namespace

hipError_t launch_quantize(const void* src, int dtype, int64_t rows, int64_t cols, int64_t ld,
                           int axis, int format, void* codes, int8_t* scales, hipStream_t s) {
    switch (format) {
        case 0: return launch_fmt<FmtE4C3>(src, dtype, rows, cols, ld, axis, 0, codes, scales, s);
        case 1: return launch_fmt<FmtE5C2>(src, dtype, rows, cols, ld, axis, 1, codes, scales, s);
        default: return launch_fmt<FmtE3C3>(src, dtype, rows, cols, ld, axis, 2, codes, scales, s);
    }
}

}  // namespace curvefp
