// CurveFP block quantization Q(X) on gfx950 (Sec. 3.1 of the CurveFP paper).
//
// For a block of G values (G a multiple of 32; 32 by default) with maximum magnitude amax:
//   scale  a = smallest integer with amax <= 2^a * fl32(L_max)  (ceil-absmax; L_max = r^{n_max/K},
//          the top level, 2^{n_max/K} with binary radix),
//          computed on the fp32 bit pattern: a = e(amax) - o_hi + [mant(amax) > mant(fl32(L_max))];
//   element: y = |x| 2^{-a} is formed exactly by subtracting a from the exponent
//          field; its rank is looked up in a per-format table indexed by the
//          bfloat16-truncated bits of y over the octaves that can reach a nonzero
//          code, plus one compare of the low 16 bits against the single decision
//          point a table bucket can hold.  The table encodes the nearest-level rule
//          (nearest in absolute error, saturating at the endpoints) derived on the host.
// Memory: HBM-bound; one pass, coalesced 16-byte loads, one byte (or 7 bits)
// per code and one byte per block written.  Blocks of 64..512 along rows take their maximum
// over the G/8 lanes that hold them; every other G first writes the block scales in a pass of
// their own (the scale rule is monotone in amax, so the scale of a block is that of its
// largest element), and the quantize pass then reads them.  Codes are laid out per 32
// elements (E3C3: 28 bytes) whatever G is.
#include "codec.hpp"
#include "curvefp_internal.hpp"
#include "device_util.hpp"
#include "planes.hpp"
#include "curvefp_tables.inc"

#include <cstring>
#include <type_traits>

namespace curvefp {

// compile-time tables (curvefp_tables.inc, written at build time by gen_tables)
__constant__ uint32_t g_qlut[NUM_FORMATS][QLUT_MAX] = CURVEFP_QLUT_INIT;
// bfloat16 sources: the low 16 bits of every scaled magnitude are zero, so the bucket's
// decision point is never passed and the rank is the bucket's base rank alone (one byte)
__constant__ __attribute__((aligned(16))) uint8_t g_qlut8[NUM_FORMATS][QLUT_MAX] = CURVEFP_QLUT8_INIT;
__constant__ uint32_t g_lmax_mant[NUM_FORMATS] = CURVEFP_LMAX_MANT_INIT;
// reconstruction tables for the static-scale search (the dequantizer's, see codec.hpp): binary
// radix 8 entries by curve index, rational radix 128 by magnitude rank
__constant__ uint32_t g_qr_mant[NUM_FORMATS][128] = CURVEFP_QR_MANT_INIT;
__constant__ uint64_t g_qr_sig[NUM_FORMATS][128] = CURVEFP_QR_SIG_INIT;
// the GEMM operands' expansion pairs (the GEMM's table, gemm.hip), for quantize-and-prepare
__constant__ uint32_t g_qp_dec[NUM_FORMATS][GEMM_DEC_ENTRIES] = CURVEFP_DEC_INIT;

namespace {

template <class F>
__device__ __forceinline__ int block_scale(uint32_t amax, uint32_t lmax_mant) {
    // an all-zero block (every integer a satisfies 0 <= 2^a fl32(L_max)) and a subnormal maximum
    // both take the bottom of the scale range
    const int ef = (int)(amax >> 23);
    if (ef == 0) return -127;
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

// the same for a yb whose low 16 bits are zero, with the one-byte table
template <class F>
__device__ __forceinline__ uint32_t rank_lookup(int32_t yb, const uint8_t* lut) {
    int32_t idx = (yb >> 16) - ((127 + F::OZ) << 7);
    if (idx < 0) return 0;
    return lut[min(idx, F::QLUT_SIZE - 1)];
}

// fast path: a >= A_FAST_MIN, where subnormal or zero inputs can only reach rank 0
template <class F, class T>
__device__ __forceinline__ uint32_t rank_fast(uint32_t mag, int a, const T* lut) {
    return rank_lookup<F>((int32_t)mag - (a << 23), lut);
}

// exact path for blocks with tiny scales: normalize subnormal inputs first
template <class F, class T>
__device__ __forceinline__ uint32_t rank_exact(uint32_t mag, int a, const T* lut) {
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

template <class F, class T>
__device__ __forceinline__ void ranks_of(const uint32_t* mag, int n, int a, const T* lut, uint32_t* r) {
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

// unpack 8 consecutive source elements into magnitude bits (as fp32) and sign bits
template <bool BF16>
__device__ __forceinline__ void unpack8(const uint4* v, uint32_t* mag, uint32_t* sgn) {
    if (BF16) {
        const uint32_t w[4] = {v[0].x, v[0].y, v[0].z, v[0].w};
#pragma unroll
        for (int i = 0; i < 4; i++) {
            mag[2 * i] = (w[i] << 16) & 0x7FFF0000u;
            mag[2 * i + 1] = w[i] & 0x7FFF0000u;
            sgn[2 * i] = (w[i] >> 15) & 1u;
            sgn[2 * i + 1] = w[i] >> 31;
        }
    } else {
        const uint32_t w[8] = {v[0].x, v[0].y, v[0].z, v[0].w, v[1].x, v[1].y, v[1].z, v[1].w};
#pragma unroll
        for (int i = 0; i < 8; i++) {
            mag[i] = w[i] & 0x7FFFFFFFu;
            sgn[i] = w[i] >> 31;
        }
    }
}

// the maximum over the 2^lgl lanes (lgl in 2..6, aligned groups, all active) that hold one
// block: DPP within 16 lanes (after the quad maximum, a half-row mirror pairs each lane with
// one of the other quad, a row mirror with one of the other half), shuffles beyond
__device__ __forceinline__ uint32_t group_max_u32(uint32_t v, int lgl) {
    v = quad_max_u32(v);
    if (lgl >= 3) v = max(v, dpp_u32<DPP_ROW_HALF_MIRROR>(v));
    if (lgl >= 4) v = max(v, dpp_u32<DPP_ROW_MIRROR>(v));
    for (int o = 16; o < (1 << lgl); o <<= 1) v = max(v, (uint32_t)__shfl_xor((int)v, o));
    return v;
}

// the codes of 8 consecutive elements (magnitudes and signs) at scale a
template <class F, class T>
__device__ __forceinline__ void chunk_codes(const uint32_t* mag, const uint32_t* sgn, int a, const T* lut,
                                            uint32_t* c) {
    uint32_t rk[8];
    ranks_of<F>(mag, 8, a, lut, rk);
#pragma unroll
    for (int i = 0; i < 8; i++) c[i] = rk[i] | ((rk[i] != 0 ? sgn[i] : 0u) << F::EC);
}

// codes c of chunk g stored at chunk g of `codes`; E3C3 packs 7 bits per code over the quad that
// holds a group of 32
template <class F, bool NTS>
__device__ __forceinline__ void store_codes(const uint32_t* c, uint32_t g, uint8_t* __restrict__ codes) {
    const int part = (int)(g & 3);
    const uint32_t b = g >> 2;   // group of 32 (groups are contiguous in the output)
    if (!F::PACKED7) {
        st8<NTS>(codes + (uint64_t)g * 8, c[0] | (c[1] << 8) | (c[2] << 16) | (c[3] << 24),
                 c[4] | (c[5] << 8) | (c[6] << 16) | (c[7] << 24));
    } else {
        // 56-bit chunk of this lane; the group's string is chunk0 | chunk1 << 56 | ...
        uint64_t chunk = 0;
#pragma unroll
        for (int i = 0; i < 8; i++) chunk |= (uint64_t)c[i] << (7 * i);
        const uint32_t nlo = dpp_u32<QP_NEXT>((uint32_t)chunk);
        const uint32_t nhi = dpp_u32<QP_NEXT>((uint32_t)(chunk >> 32));
        const uint64_t next = ((uint64_t)nhi << 32) | nlo;
        uint32_t* base = reinterpret_cast<uint32_t*>(codes + (uint64_t)b * 28);
        if (part < 3) {
            const uint64_t lo64 = chunk | (next << 56);
            const uint64_t hi64 = next >> 8;
            const int sh = 8 * part;
            const uint64_t w = sh ? ((lo64 >> sh) | (hi64 << (64 - sh))) : lo64;
            st4<NTS>(base + 2 * part, (uint32_t)w);
            st4<NTS>(base + 2 * part + 1, (uint32_t)(w >> 32));
        } else {
            st4<NTS>(base + 6, (uint32_t)(chunk >> 24));
        }
    }
}

// codes of chunk g (8 consecutive elements, magnitudes and signs) at scale a, stored at chunk g
// of `codes`
template <class F, bool NTS, class T>
__device__ __forceinline__ void encode_chunk(const uint32_t* mag, const uint32_t* sgn, int a, uint32_t g,
                                             const T* lut, uint8_t* __restrict__ codes) {
    uint32_t c[8];
    chunk_codes<F>(mag, sgn, a, lut, c);
    store_codes<F, NTS>(c, g, codes);
}

// quantize one chunk of 8 consecutive elements; 2^lgl consecutive lanes hold one block of
// 8 * 2^lgl elements (a quad for 32).  lgl < 0: the block scales were written by the scale
// pass, scale of chunk g at g / (G / 8) (dgl)
template <class F, bool BF16, bool NTS, class T>
__device__ __forceinline__ void quantize_chunk(const uint4* v, uint32_t g, const T* lut,
                                               uint32_t lmax_mant, uint8_t* __restrict__ codes,
                                               int8_t* __restrict__ scales, int lgl, Div32 dgl) {
    uint32_t mag[8], sgn[8];
    unpack8<BF16>(v, mag, sgn);
    int a;
    if (lgl >= 0) {
        uint32_t amax = 0;
#pragma unroll
        for (int i = 0; i < 8; i++) amax = max(amax, mag[i]);
        amax = lgl == 2 ? quad_max_u32(amax) : group_max_u32(amax, lgl);
        a = scale_of<F>(amax, lmax_mant);
    } else {
        a = scales[div32(g, dgl)];
    }
    encode_chunk<F, NTS>(mag, sgn, a, g, lut, codes);
    if (lgl >= 0 && (g & ((1u << lgl) - 1)) == 0) scales[g >> lgl] = (int8_t)a;
}

// blocks along rows: chunk g (8 elements) is chunk g mod cpr of row g / cpr; four consecutive
// chunks form a block.  Each thread has U chunks in flight, 256 chunks apart, so every load
// instruction of a wave reads one contiguous span.
template <class F, bool BF16, int U, bool NT, bool NTS>
__global__ __launch_bounds__(256) void quantize_rows_kernel(
    const void* __restrict__ src, uint32_t nchunks, uint32_t cpr, Div32 dcpr, int64_t ld,
    uint8_t* __restrict__ codes, int8_t* __restrict__ scales, int fidx, int lgl, Div32 dgl) {
    using T = typename std::conditional<BF16, uint8_t, uint32_t>::type;
    __shared__ __attribute__((aligned(16))) T lut[F::QLUT_SIZE];
    constexpr int ESZ = BF16 ? 2 : 4;
    constexpr int NV = BF16 ? 1 : 2;   // 16-byte loads per chunk
    const bool dense = ld == (int64_t)cpr * 8;
    const char* s8 = reinterpret_cast<const char*>(src);
    auto load = [&](uint32_t g0, uint4 (*v)[NV]) {
#pragma unroll
        for (int u = 0; u < U; u++) {
            const uint32_t g = g0 + 256u * u;
            if (g < nchunks) {
                int64_t e;
                if (dense) {
                    e = (int64_t)g * 8;
                } else {
                    const uint32_t r = div32(g, dcpr);
                    e = (int64_t)r * ld + (int64_t)(g - r * cpr) * 8;
                }
                const uint4* p = reinterpret_cast<const uint4*>(s8 + e * ESZ);
#pragma unroll
                for (int t = 0; t < NV; t++) v[u][t] = ld16<NT>(p + t);
            }
        }
    };
    const uint32_t step = gridDim.x * (256u * U);
    uint32_t g0 = blockIdx.x * (256u * U) + threadIdx.x;
    // the first chunks are requested before the table is filled, so both latencies overlap
    uint4 v[U][NV];
    load(g0, v);
    if (BF16) {
        const uint32_t* s32 = reinterpret_cast<const uint32_t*>(g_qlut8[fidx]);
        uint32_t* l32 = reinterpret_cast<uint32_t*>(lut);
        for (int i = threadIdx.x; i < F::QLUT_SIZE / 4; i += blockDim.x) l32[i] = s32[i];
    } else {
        for (int i = threadIdx.x; i < F::QLUT_SIZE; i += blockDim.x) lut[i] = (T)g_qlut[fidx][i];
    }
    const uint32_t lmax_mant = g_lmax_mant[fidx];
    __syncthreads();

    while (g0 < nchunks) {
        // next chunks in flight while these are quantized
        const uint32_t g1 = g0 + step;
        uint4 w[U][NV];
        const bool more = g1 < nchunks && g1 > g0;
        if (more) load(g1, w);
#pragma unroll
        for (int u = 0; u < U; u++) {
            const uint32_t g = g0 + 256u * u;
            if (g < nchunks) quantize_chunk<F, BF16, NTS>(v[u], g, lut, lmax_mant, codes, scales, lgl, dgl);
        }
        if (!more) break;
#pragma unroll
        for (int u = 0; u < U; u++)
#pragma unroll
            for (int t = 0; t < NV; t++) v[u][t] = w[u][t];
        g0 = g1;
    }
}

// quantize-transpose: thread g takes column g mod cols and R consecutive blocks of 32 rows
// (row group g / cols), so the loads of a wave read one contiguous span of a source row and
// each thread writes R * 32 contiguous code bytes (R * 28 for E3C3) and R scales.  given != 0:
// blocks of G rows whose scales the scale pass wrote, [cols][nsb], 32-row block rb in G-block
// rb / (G / 32) (dgq)
template <class F, bool BF16, int R>
__global__ __launch_bounds__(256) void quantize_cols_kernel(
    const void* __restrict__ src, uint32_t nthreads, uint32_t cols, Div32 dcols, int64_t rows, int64_t ld,
    uint8_t* __restrict__ codes, int8_t* __restrict__ scales, int fidx, int given, int64_t nsb, Div32 dgq) {
    __shared__ uint32_t lut[F::QLUT_SIZE];
    for (int i = threadIdx.x; i < F::QLUT_SIZE; i += blockDim.x) lut[i] = g_qlut[fidx][i];
    const uint32_t lmax_mant = g_lmax_mant[fidx];
    __syncthreads();

    const uint32_t g = blockIdx.x * 256u + threadIdx.x;
    if (g >= nthreads) return;
    const uint32_t rg = div32(g, dcols);
    const uint32_t c = g - rg * cols;
    const int64_t rblocks = rows / 32;
#pragma unroll 1
    for (int t = 0; t < R; t++) {
        const int64_t rb = (int64_t)rg * R + t;
        uint32_t mag[32], sgn[32];
#pragma unroll
        for (int i = 0; i < 32; i++) {
            const int64_t e = (rb * 32 + i) * ld + c;
            const uint32_t w = BF16 ? ((uint32_t)reinterpret_cast<const uint16_t*>(src)[e] << 16)
                                    : reinterpret_cast<const uint32_t*>(src)[e];
            mag[i] = w & 0x7FFFFFFFu;
            sgn[i] = w >> 31;
        }
        int a;
        if (given) {
            a = scales[(int64_t)c * nsb + div32((uint32_t)rb, dgq)];
        } else {
            uint32_t amax = 0;
#pragma unroll
            for (int i = 0; i < 32; i++) amax = max(amax, mag[i]);
            a = scale_of<F>(amax, lmax_mant);
        }
        uint32_t rk[32];
        ranks_of<F>(mag, 32, a, lut, rk);
        uint32_t cc[32];
#pragma unroll
        for (int i = 0; i < 32; i++) cc[i] = rk[i] | ((rk[i] != 0 ? sgn[i] : 0u) << F::EC);
        if (!F::PACKED7) {
            uint8_t* o = codes + (int64_t)c * rows + rb * 32;
#pragma unroll
            for (int q = 0; q < 2; q++) {
                const uint32_t* k = cc + 16 * q;
                st16<true>(o + 16 * q, k[0] | (k[1] << 8) | (k[2] << 16) | (k[3] << 24),
                           k[4] | (k[5] << 8) | (k[6] << 16) | (k[7] << 24),
                           k[8] | (k[9] << 8) | (k[10] << 16) | (k[11] << 24),
                           k[12] | (k[13] << 8) | (k[14] << 16) | (k[15] << 24));
            }
        } else {
            uint32_t w[7] = {0, 0, 0, 0, 0, 0, 0};
#pragma unroll
            for (int i = 0; i < 32; i++) {
                const int bit = 7 * i, d = bit >> 5, sh = bit & 31;
                w[d] |= cc[i] << sh;
                if (sh > 25) w[d + 1] |= cc[i] >> (32 - sh);
            }
            uint32_t* o = reinterpret_cast<uint32_t*>(codes + ((int64_t)c * rblocks + rb) * 28);
#pragma unroll
            for (int d = 0; d < 7; d++) st4<true>(o + d, w[d]);
        }
        if (!given) scales[(int64_t)c * rblocks + rb] = (int8_t)a;
    }
}

// Scale pass (blocks the quantize kernels cannot reduce in one pass): the ceil-absmax scale of
// every block of G elements.  Blocks along rows: one wave per block, 16-byte loads.
template <class F, bool BF16>
__global__ __launch_bounds__(256) void block_scales_rows_kernel(const void* __restrict__ src, int64_t nblocks,
                                                                int64_t bpr, int64_t ld, int G,
                                                                int8_t* __restrict__ scales, int fidx) {
    constexpr int ESZ = BF16 ? 2 : 4;
    constexpr int NV = BF16 ? 1 : 2;   // 16-byte loads per chunk of 8 elements
    const int64_t blk = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    const int lane = (int)(threadIdx.x & 63);
    if (blk >= nblocks) return;        // whole waves
    const int64_t r = blk / bpr, cb = blk - r * bpr;
    const uint4* p = reinterpret_cast<const uint4*>(reinterpret_cast<const char*>(src) + (r * ld + cb * G) * ESZ);
    uint32_t amax = 0;
#pragma unroll 4
    for (int c = lane; c < G / 8; c += 64) {
        uint4 v[NV];
#pragma unroll
        for (int t = 0; t < NV; t++) v[t] = ld16<false>(p + NV * c + t);
        uint32_t mag[8], sgn[8];
        unpack8<BF16>(v, mag, sgn);
#pragma unroll
        for (int i = 0; i < 8; i++) amax = max(amax, mag[i]);
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) amax = max(amax, (uint32_t)__shfl_xor((int)amax, o));
    if (lane == 0) scales[blk] = (int8_t)scale_of<F>(amax, g_lmax_mant[fidx]);
}

// blocks along columns (quantize-transpose): a workgroup takes 64 columns of one block of G
// rows, in four row parts; scales [cols][rows / G]
template <class F, bool BF16>
__global__ __launch_bounds__(256) void block_scales_cols_kernel(const void* __restrict__ src, int64_t rows,
                                                                int64_t cols, int64_t ld, int G, int64_t ncg,
                                                                int8_t* __restrict__ scales, int fidx) {
    __shared__ uint32_t red[256];
    const int t = (int)threadIdx.x, j = t & 63, part = t >> 6;
    const int64_t b = (int64_t)blockIdx.x / ncg, cg = (int64_t)blockIdx.x - b * ncg;
    const int64_t c = cg * 64 + j;
    uint32_t amax = 0;
    if (c < cols) {
#pragma unroll 8
        for (int i = part; i < G; i += 4) {
            const int64_t e = (b * G + i) * ld + c;
            const uint32_t w = BF16 ? ((uint32_t)reinterpret_cast<const uint16_t*>(src)[e] << 16)
                                    : reinterpret_cast<const uint32_t*>(src)[e];
            amax = max(amax, w & 0x7FFFFFFFu);
        }
    }
    red[t] = amax;
    __syncthreads();
    if (t < 64 && c < cols) {
        const uint32_t m = max(max(red[t], red[t + 64]), max(red[t + 128], red[t + 192]));
        scales[c * (rows / G) + b] = (int8_t)scale_of<F>(m, g_lmax_mant[fidx]);
    }
}

template <class F, bool BF16, int U>
hipError_t launch_rows_u(const void* src, int64_t rows, int64_t cols, int64_t ld, int fidx, uint8_t* codes,
                         int8_t* scales, int block, int lgl, Div32 dgl, hipStream_t s) {
    const int64_t cpr = cols / 8;
    // 32-bit chunk indices: slabs of at most 2^31 chunks
    const int64_t slab = ((int64_t)1 << 31) / cpr;
    for (int64_t r0 = 0; r0 < rows; r0 += slab) {
        const int64_t nr = rows - r0 < slab ? rows - r0 : slab;
        const int64_t nchunks = nr * cpr;
        int64_t blocks = (nchunks + 256 * U - 1) / (256 * U);
        blocks = blocks < 32768 ? blocks : 32768;
        const void* sp = reinterpret_cast<const char*>(src) + r0 * ld * (BF16 ? 2 : 4);
        uint8_t* cp = codes + (F::PACKED7 ? r0 * (cols / 32) * 28 : r0 * cols);
        int8_t* scp = scales + r0 * (cols / block);
        hipLaunchKernelGGL((quantize_rows_kernel<F, BF16, U, true, true>), dim3(blocks), dim3(256), 0, s, sp,
                           (uint32_t)nchunks, (uint32_t)cpr, make_div32((uint32_t)cpr), ld, cp, scp, fidx, lgl, dgl);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

// bf16 sources: two chunks (32 bytes) in flight per thread at every size.  Measured against eight
// and one on 8192 x 4096, 14336 x 4096, 16384 x 8192, 32768 x 8192 and 32768 x 16384 sources, calls
// alternating in one process: eight 6-9% slower on all but 16384 x 8192 (2.5%), one 10-20% slower.
// fp32 sources: 64 bytes per thread from 2048 workgroups on, 32 below, so that smaller tensors
// still spread over every compute unit.  Blocks of 32..512 (a power of two) are reduced over their
// lanes; any other block size runs the scale pass first.
template <class F, bool BF16>
hipError_t launch_rows(const void* src, int64_t rows, int64_t cols, int64_t ld, int fidx, uint8_t* codes,
                       int8_t* scales, int block, hipStream_t s) {
    int lgl = -1;
    if (block <= 512 && (block & (block - 1)) == 0)
        for (lgl = 0; (8 << lgl) < block; lgl++) {}
    const Div32 dgl = make_div32((uint32_t)(block / 8));
    if (lgl < 0) {
        const int64_t nb = rows * (cols / block);
        hipLaunchKernelGGL((block_scales_rows_kernel<F, BF16>), dim3((unsigned)((nb + 3) / 4)), dim3(256), 0, s, src,
                           nb, cols / block, ld, block, scales, fidx);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    const int64_t nchunks = rows * (cols / 8);
    if (BF16 || nchunks >= (int64_t)2048 * 256 * 2)
        return launch_rows_u<F, BF16, 2>(src, rows, cols, ld, fidx, codes, scales, block, lgl, dgl, s);
    return launch_rows_u<F, BF16, 1>(src, rows, cols, ld, fidx, codes, scales, block, lgl, dgl, s);
}

// quantize-transpose through LDS: a workgroup takes 128 rows (four blocks) x 64 columns.  The
// tile is read with 16-byte loads along the source rows, each thread then quantizes one
// column's group of 32 from LDS (a wave reads one contiguous row segment per step; for blocks
// of G > 32 rows the scale pass has written the block scales), and the
// codes go back through LDS so every column's 128 code bytes (112 for E3C3) leave as whole
// 16-byte stores.  Needs rows % 128 == 0, cols % 8 == 0 and a 16-byte aligned source.
constexpr int TT_ROWS = 128, TT_COLS = 64;
constexpr int TT_OUT_STRIDE = 144;   // 128 code bytes + 16: the 16-byte writes of a wave spread over the banks

template <class F, bool BF16>
__global__ __launch_bounds__(256) void quantize_cols_tiled_kernel(
    const void* __restrict__ src, int64_t rows, int64_t cols, int64_t ld,
    uint8_t* __restrict__ codes, int8_t* __restrict__ scales, int fidx, int given, int64_t nsb, Div32 dgq) {
    using T = typename std::conditional<BF16, uint8_t, uint32_t>::type;
    constexpr int ESZ = BF16 ? 2 : 4;
    constexpr int SEG = TT_COLS * ESZ / 16;            // 16-byte pieces per tile row
    __shared__ __attribute__((aligned(16))) T lut[F::QLUT_SIZE];
    __shared__ __attribute__((aligned(16))) char tile[TT_ROWS * TT_COLS * ESZ];
    __shared__ __attribute__((aligned(16))) uint8_t outb[TT_COLS * TT_OUT_STRIDE];
    __shared__ int8_t scl[TT_COLS * 4];

    const int tid = threadIdx.x;
    const int64_t c0 = (int64_t)blockIdx.x * TT_COLS, r0 = (int64_t)blockIdx.y * TT_ROWS;
    const char* s8 = reinterpret_cast<const char*>(src);
    // phase 1: the tile, 16 bytes per load (columns past the end are not read)
    uint4 v[TT_ROWS * SEG / 256];
#pragma unroll
    for (int k = 0; k < TT_ROWS * SEG / 256; k++) {
        const int piece = tid + 256 * k, row = piece / SEG, seg = piece % SEG;
        const int64_t col = c0 + seg * (16 / ESZ);
        v[k] = col < cols ? ld16<true>(reinterpret_cast<const uint4*>(s8 + ((r0 + row) * ld + col) * ESZ))
                          : make_uint4(0, 0, 0, 0);
    }
    if (BF16) {
        const uint32_t* s32 = reinterpret_cast<const uint32_t*>(g_qlut8[fidx]);
        uint32_t* l32 = reinterpret_cast<uint32_t*>(lut);
        for (int i = tid; i < F::QLUT_SIZE / 4; i += 256) l32[i] = s32[i];
    } else {
        for (int i = tid; i < F::QLUT_SIZE; i += 256) lut[i] = (T)g_qlut[fidx][i];
    }
    const uint32_t lmax_mant = g_lmax_mant[fidx];
#pragma unroll
    for (int k = 0; k < TT_ROWS * SEG / 256; k++)
        *reinterpret_cast<uint4*>(tile + (tid + 256 * k) * 16) = v[k];
    __syncthreads();

    // phase 2: thread = (column j, block b)
    const int j = tid & (TT_COLS - 1), b = tid >> 6;
    uint32_t mag[32], sgn[32];
#pragma unroll
    for (int i = 0; i < 32; i++) {
        const int e = (b * 32 + i) * TT_COLS + j;
        const uint32_t w = BF16 ? ((uint32_t)reinterpret_cast<const uint16_t*>(tile)[e] << 16)
                                : reinterpret_cast<const uint32_t*>(tile)[e];
        mag[i] = w & 0x7FFFFFFFu;
        sgn[i] = w >> 31;
    }
    int a = 0;
    if (given) {
        if (c0 + j < cols) a = scales[(c0 + j) * nsb + div32((uint32_t)(r0 / 32 + b), dgq)];
    } else {
        uint32_t amax = 0;
#pragma unroll
        for (int i = 0; i < 32; i++) amax = max(amax, mag[i]);
        a = scale_of<F>(amax, lmax_mant);
    }
    uint32_t rk[32];
    ranks_of<F>(mag, 32, a, lut, rk);
    uint32_t cc[32];
#pragma unroll
    for (int i = 0; i < 32; i++) cc[i] = rk[i] | ((rk[i] != 0 ? sgn[i] : 0u) << F::EC);
    uint8_t* ob = outb + j * TT_OUT_STRIDE;
    if (!F::PACKED7) {
#pragma unroll
        for (int q = 0; q < 2; q++) {
            const uint32_t* k = cc + 16 * q;
            *reinterpret_cast<uint4*>(ob + b * 32 + 16 * q) =
                make_uint4(k[0] | (k[1] << 8) | (k[2] << 16) | (k[3] << 24),
                           k[4] | (k[5] << 8) | (k[6] << 16) | (k[7] << 24),
                           k[8] | (k[9] << 8) | (k[10] << 16) | (k[11] << 24),
                           k[12] | (k[13] << 8) | (k[14] << 16) | (k[15] << 24));
        }
    } else {
        uint32_t w[7] = {0, 0, 0, 0, 0, 0, 0};
#pragma unroll
        for (int i = 0; i < 32; i++) {
            const int bit = 7 * i, d = bit >> 5, sh = bit & 31;
            w[d] |= cc[i] << sh;
            if (sh > 25) w[d + 1] |= cc[i] >> (32 - sh);
        }
#pragma unroll
        for (int d = 0; d < 7; d++) *reinterpret_cast<uint32_t*>(ob + b * 28 + 4 * d) = w[d];
    }
    scl[j * 4 + b] = (int8_t)a;
    __syncthreads();

    // phase 3: each column's code bytes for the four blocks are contiguous in the output
    constexpr int CB = F::PACKED7 ? 4 * 28 : 128;   // code bytes per column and tile
    const int64_t rblocks = rows / 32;
#pragma unroll
    for (int k = 0; k < (TT_COLS * CB / 16 + 255) / 256; k++) {
        const int piece = tid + 256 * k;
        if (piece < TT_COLS * CB / 16) {
            const int jj = piece / (CB / 16), qq = piece % (CB / 16);
            const int64_t col = c0 + jj;
            if (col < cols) {
                const uint4 x = *reinterpret_cast<const uint4*>(outb + jj * TT_OUT_STRIDE + 16 * qq);
                uint8_t* dst = F::PACKED7 ? codes + (col * rblocks + r0 / 32) * 28 : codes + col * rows + r0;
                st16<true>(dst + 16 * qq, x.x, x.y, x.z, x.w);
            }
        }
    }
    if (!given) {
        const int jj = tid >> 2, bb = tid & 3;
        if (c0 + jj < cols) scales[(c0 + jj) * rblocks + r0 / 32 + bb] = scl[jj * 4 + bb];
    }
}

// given != 0: the block scales (blocks of `block` rows) are already in `scales`
template <class F, int R>
hipError_t launch_cols(const void* src, int dtype, int64_t rows, int64_t cols, int64_t ld, int fidx,
                       uint8_t* codes, int8_t* scales, int block, int given, hipStream_t s) {
    const Div32 dgq = make_div32((uint32_t)(block / 32));
    // column slabs keep the thread count of one launch below 2^31
    const int64_t groups = rows / (32 * R);
    const int64_t slab = ((int64_t)1 << 31) / groups;
    for (int64_t c0 = 0; c0 < cols; c0 += slab) {
        const int64_t nc = cols - c0 < slab ? cols - c0 : slab;
        const int64_t nthreads = groups * nc;
        const int64_t blocks = (nthreads + 255) / 256;
        const int64_t esz = dtype == 1 ? 2 : 4;
        const void* sp = reinterpret_cast<const char*>(src) + c0 * esz;
        uint8_t* cp = codes + (F::PACKED7 ? c0 * (rows / 32) * 28 : c0 * rows);
        int8_t* scp = scales + c0 * (rows / block);
        if (dtype == 1)
            hipLaunchKernelGGL((quantize_cols_kernel<F, true, R>), dim3((unsigned)blocks), dim3(256), 0, s, sp,
                               (uint32_t)nthreads, (uint32_t)nc, make_div32((uint32_t)nc), rows, ld, cp, scp, fidx,
                               given, rows / block, dgq);
        else
            hipLaunchKernelGGL((quantize_cols_kernel<F, false, R>), dim3((unsigned)blocks), dim3(256), 0, s, sp,
                               (uint32_t)nthreads, (uint32_t)nc, make_div32((uint32_t)nc), rows, ld, cp, scp, fidx,
                               given, rows / block, dgq);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

template <class F>
hipError_t launch_fmt(const void* src, int dtype, int64_t rows, int64_t cols, int64_t ld, int axis,
                      int fidx, int block, void* codes, int8_t* scales, hipStream_t s) {
    uint8_t* cp = reinterpret_cast<uint8_t*>(codes);
    if (axis == 1) {
        return dtype == 1 ? launch_rows<F, true>(src, rows, cols, ld, fidx, cp, scales, block, s)
                          : launch_rows<F, false>(src, rows, cols, ld, fidx, cp, scales, block, s);
    }
    // blocks of more than 32 rows: scale pass, then the quantize-transpose reads the scales
    const int given = block > 32;
    const Div32 dgq = make_div32((uint32_t)(block / 32));
    if (given) {
        const int64_t ncg = (cols + 63) / 64;
        const dim3 grid((unsigned)(ncg * (rows / block)));
        if (dtype == 1)
            hipLaunchKernelGGL((block_scales_cols_kernel<F, true>), grid, dim3(256), 0, s, src, rows, cols, ld, block,
                               ncg, scales, fidx);
        else
            hipLaunchKernelGGL((block_scales_cols_kernel<F, false>), grid, dim3(256), 0, s, src, rows, cols, ld, block,
                               ncg, scales, fidx);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    const int64_t esz = dtype == 1 ? 2 : 4;
    const bool tiled = rows % TT_ROWS == 0 && cols % 8 == 0 && (reinterpret_cast<uintptr_t>(src) & 15) == 0 &&
                       (ld * esz) % 16 == 0 && rows / TT_ROWS <= 65535;
    if (tiled) {
        const dim3 grid((unsigned)((cols + TT_COLS - 1) / TT_COLS), (unsigned)(rows / TT_ROWS));
        if (dtype == 1)
            hipLaunchKernelGGL((quantize_cols_tiled_kernel<F, true>), grid, dim3(256), 0, s, src, rows, cols, ld, cp,
                               scales, fidx, given, rows / block, dgq);
        else
            hipLaunchKernelGGL((quantize_cols_tiled_kernel<F, false>), grid, dim3(256), 0, s, src, rows, cols, ld, cp,
                               scales, fidx, given, rows / block, dgq);
        return hipGetLastError();
    }
    return launch_cols<F, 1>(src, dtype, rows, cols, ld, fidx, cp, scales, block, given, s);
}

// ---------------------------------------------------------------------------------------------
// S-bit scale exponents (Eq. effective-rate with an S-bit scale field).  One workgroup per row:
// pass 1 writes the row's maxima per group of 32 to LDS; the block scales follow, the row's
// reference (the largest scale among its finite blocks that are not all zero, 0 if none), and
// every block's scale is raised to at least reference - (2^S - 2); pass 2 reads the row again
// (from the caches) and quantizes it at those scales.  The offsets reference - scale (2^S - 1
// for a block that held a NaN or an infinity, 0 for an all-zero block) leave packed S bits
// each, LSB first, each row padded to whole bytes.
constexpr int COMPACT_MAX_GROUPS = 4096;   // up to 131072 elements per row
constexpr int COMPACT_NONE = -1000;         // below every scale

template <class F, bool BF16>
__global__ __launch_bounds__(256) void quantize_compact_kernel(const void* __restrict__ src, int64_t cols, int64_t ld,
                                                               int G, int S, uint8_t* __restrict__ codes,
                                                               int8_t* __restrict__ row_ref,
                                                               uint8_t* __restrict__ offsets, int64_t off_bytes,
                                                               int fidx) {
    using T = typename std::conditional<BF16, uint8_t, uint32_t>::type;
    constexpr int ESZ = BF16 ? 2 : 4;
    constexpr int NV = BF16 ? 1 : 2;
    __shared__ __attribute__((aligned(16))) T lut[F::QLUT_SIZE];
    __shared__ uint32_t gmax[COMPACT_MAX_GROUPS];
    __shared__ int bsc[COMPACT_MAX_GROUPS];
    __shared__ uint8_t doff[COMPACT_MAX_GROUPS];
    __shared__ int wred[4];
    const int tid = (int)threadIdx.x;
    const int64_t row = blockIdx.x;
    const uint4* p = reinterpret_cast<const uint4*>(reinterpret_cast<const char*>(src) + row * ld * ESZ);
    const int nchunks = (int)(cols / 8), nb = (int)(cols / G), gpb = G / 32;
    if (BF16) {
        const uint32_t* s32 = reinterpret_cast<const uint32_t*>(g_qlut8[fidx]);
        uint32_t* l32 = reinterpret_cast<uint32_t*>(lut);
        for (int i = tid; i < F::QLUT_SIZE / 4; i += 256) l32[i] = s32[i];
    } else {
        for (int i = tid; i < F::QLUT_SIZE; i += 256) lut[i] = (T)g_qlut[fidx][i];
    }
    const uint32_t lmax_mant = g_lmax_mant[fidx];
    // pass 1: group maxima (the four chunks of a group sit in one quad of lanes)
    for (int c = tid; c < nchunks; c += 256) {
        uint4 v[NV];
#pragma unroll
        for (int t = 0; t < NV; t++) v[t] = ld16<false>(p + NV * c + t);
        uint32_t mag[8], sgn[8];
        unpack8<BF16>(v, mag, sgn);
        uint32_t amax = 0;
#pragma unroll
        for (int i = 0; i < 8; i++) amax = max(amax, mag[i]);
        amax = quad_max_u32(amax);
        if ((c & 3) == 0) gmax[c >> 2] = amax;
    }
    __syncthreads();
    // block scales and the row's reference
    int lm = COMPACT_NONE;
    for (int b = tid; b < nb; b += 256) {
        uint32_t m = 0;
        for (int j = 0; j < gpb; j++) m = max(m, gmax[b * gpb + j]);
        const int a = scale_of<F>(m, lmax_mant);
        bsc[b] = m == 0 ? COMPACT_NONE : a;          // all-zero blocks take no part
        if (m != 0 && a != -128) lm = max(lm, a);
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) lm = max(lm, __shfl_xor(lm, o));
    if ((tid & 63) == 0) wred[tid >> 6] = lm;
    __syncthreads();
    const int top = max(max(wred[0], wred[1]), max(wred[2], wred[3]));
    const int ref = top == COMPACT_NONE ? 0 : top;
    const int window = (1 << S) - 2;
    for (int b = tid; b < nb; b += 256) {
        const int a = bsc[b];
        int ae, d;
        if (a == COMPACT_NONE) { ae = ref; d = 0; }                        // all zero
        else if (a == -128) { ae = -128; d = window + 1; }                 // NaN / Inf
        else { ae = max(a, ref - window); d = ref - ae; }
        bsc[b] = ae;
        doff[b] = (uint8_t)d;
    }
    __syncthreads();
    // pass 2: the row at its blocks' scales
    uint8_t* rc = codes + (F::PACKED7 ? row * (cols / 32) * 28 : row * cols);
    for (int c = tid; c < nchunks; c += 256) {
        uint4 v[NV];
#pragma unroll
        for (int t = 0; t < NV; t++) v[t] = ld16<false>(p + NV * c + t);
        uint32_t mag[8], sgn[8];
        unpack8<BF16>(v, mag, sgn);
        encode_chunk<F, false>(mag, sgn, bsc[(8 * c) / G], (uint32_t)c, lut, rc);
    }
    // the offsets, one output byte per thread and step
    uint8_t* ro = offsets + row * off_bytes;
    for (int64_t j = tid; j < off_bytes; j += 256) {
        uint32_t v = 0;
        for (int bit = 0; bit < 8; bit++) {
            const int64_t gb = 8 * j + bit;
            const int64_t blk = gb / S;
            if (blk < nb) v |= (uint32_t)((doff[blk] >> (gb - blk * S)) & 1) << bit;
        }
        ro[j] = (uint8_t)v;
    }
    if (tid == 0) row_ref[row] = (int8_t)ref;
}

// int8 block scales from S-bit offsets: reference - offset, -128 for the marker 2^S - 1
__global__ __launch_bounds__(256) void scales_unpack_kernel(const int8_t* __restrict__ row_ref,
                                                            const uint8_t* __restrict__ offsets, int64_t rows,
                                                            int64_t nb, int64_t off_bytes, int S,
                                                            int8_t* __restrict__ scales) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= rows * nb) return;
    const int64_t r = i / nb, b = i - r * nb;
    const uint8_t* ro = offsets + r * off_bytes;
    const int64_t gb = b * S;
    uint32_t w = ro[gb >> 3];
    if ((gb & 7) + S > 8) w |= (uint32_t)ro[(gb >> 3) + 1] << 8;
    const int d = (int)((w >> (gb & 7)) & ((1u << S) - 1));
    scales[i] = (int8_t)(d == (1 << S) - 1 ? -128 : (int)row_ref[r] - d);
}

// Tensorwise scales: one ceil-absmax scale for the whole tensor.  A 4-byte workspace word is
// cleared, every workgroup folds the largest magnitude bits it reads into it (atomicMax on the
// fp32 bit pattern: non-negative floats order as integers, NaN above infinity), the scale is
// written once per output row (the rowwise layout, all entries equal), and the quantize kernels
// then read it as the scale of a block spanning the whole blocked extent.
__global__ void tensor_max_clear_kernel(uint32_t* __restrict__ word) { *word = 0u; }

// VEC: rows 16-byte aligned with cols % 8 == 0, read in chunks of 8 elements (n = rows * cols / 8
// chunks, row of chunk g = g / (cols / 8)); otherwise one element at a time (n = rows * cols).
// n < 2^32 either way (the launcher checks).
template <bool BF16, bool VEC>
__global__ __launch_bounds__(256) void tensor_max_kernel(const void* __restrict__ src, uint32_t n, uint32_t per_row,
                                                         Div32 dpr, int64_t ld, uint32_t* __restrict__ word) {
    constexpr int ESZ = BF16 ? 2 : 4;
    constexpr int NV = BF16 ? 1 : 2;
    uint32_t m = 0;
    // four units in flight per thread: the grid is small (every workgroup ends in one atomic on
    // the same word, and those serialize), so each thread streams many units
#pragma unroll 4
    for (uint32_t g = blockIdx.x * 256u + threadIdx.x; g < n; g += gridDim.x * 256u) {
        const uint32_t r = div32(g, dpr), c = g - r * per_row;
        if (VEC) {
            const uint4* p = reinterpret_cast<const uint4*>(reinterpret_cast<const char*>(src) +
                                                            ((int64_t)r * ld + 8 * (int64_t)c) * ESZ);
            uint4 v[NV];
#pragma unroll
            for (int t = 0; t < NV; t++) v[t] = ld16<true>(p + t);
            uint32_t mag[8], sgn[8];
            unpack8<BF16>(v, mag, sgn);
#pragma unroll
            for (int i = 0; i < 8; i++) m = max(m, mag[i]);
        } else {
            const char* p = reinterpret_cast<const char*>(src) + ((int64_t)r * ld + c) * ESZ;
            const uint32_t w = BF16 ? ((uint32_t)*reinterpret_cast<const uint16_t*>(p) << 16)
                                    : *reinterpret_cast<const uint32_t*>(p);
            m = max(m, w & 0x7FFFFFFFu);
        }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) m = max(m, (uint32_t)__shfl_xor((int)m, o));
    __shared__ uint32_t wm[4];
    if ((threadIdx.x & 63) == 0) wm[threadIdx.x >> 6] = m;
    __syncthreads();
    if (threadIdx.x == 0) atomicMax(word, max(max(wm[0], wm[1]), max(wm[2], wm[3])));
}

template <class F>
__global__ __launch_bounds__(256) void tensor_scale_kernel(const uint32_t* __restrict__ word, int64_t outer,
                                                           int8_t* __restrict__ scales, int fidx) {
    const int a = scale_of<F>(*word, g_lmax_mant[fidx]);
    for (int64_t r = (int64_t)blockIdx.x * 256 + threadIdx.x; r < outer; r += (int64_t)gridDim.x * 256)
        scales[r] = (int8_t)a;
}

template <class F>
hipError_t launch_tensorwise_fmt(const void* src, int dtype, int64_t rows, int64_t cols, int64_t ld, int axis,
                                 int fidx, void* codes, int8_t* scales, uint32_t* word, hipStream_t s) {
    hipLaunchKernelGGL(tensor_max_clear_kernel, dim3(1), dim3(1), 0, s, word);
    const int64_t esz0 = dtype == 1 ? 2 : 4;
    const bool vec = cols % 8 == 0 && (reinterpret_cast<uintptr_t>(src) & 15) == 0 && (ld * esz0) % 16 == 0;
    const int64_t per_row = vec ? cols / 8 : cols;
    // slabs of rows keep the unit count of one launch at most 2^32 - 2^21, so the grid-stride
    // index (stride at most 2^20) never wraps; per_row < 2^31 (checked by the caller)
    const int64_t slab = (((int64_t)1 << 32) - ((int64_t)1 << 21)) / per_row;
    for (int64_t r0 = 0; r0 < rows; r0 += slab) {
        const int64_t nr = rows - r0 < slab ? rows - r0 : slab;
        const uint32_t n = (uint32_t)(nr * per_row);
        int64_t g = ((int64_t)n + 255) / 256;
        g = g < 256 ? g : 256;                 // one workgroup per compute unit, 256 atomics
        const void* sp = reinterpret_cast<const char*>(src) + r0 * ld * esz0;
        const Div32 dpr = make_div32((uint32_t)per_row);
        if (dtype == 1) {
            if (vec) hipLaunchKernelGGL((tensor_max_kernel<true, true>), dim3((unsigned)g), dim3(256), 0, s, sp, n,
                                        (uint32_t)per_row, dpr, ld, word);
            else hipLaunchKernelGGL((tensor_max_kernel<true, false>), dim3((unsigned)g), dim3(256), 0, s, sp, n,
                                    (uint32_t)per_row, dpr, ld, word);
        } else {
            if (vec) hipLaunchKernelGGL((tensor_max_kernel<false, true>), dim3((unsigned)g), dim3(256), 0, s, sp, n,
                                        (uint32_t)per_row, dpr, ld, word);
            else hipLaunchKernelGGL((tensor_max_kernel<false, false>), dim3((unsigned)g), dim3(256), 0, s, sp, n,
                                    (uint32_t)per_row, dpr, ld, word);
        }
    }
    const int64_t outer = axis == 1 ? rows : cols;
    int64_t gs = (outer + 255) / 256;
    gs = gs < 1024 ? gs : 1024;
    hipLaunchKernelGGL((tensor_scale_kernel<F>), dim3((unsigned)gs), dim3(256), 0, s, word, outer, scales, fidx);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    // the quantize pass with the scale given, one block per output row of the blocked extent
    uint8_t* cp = reinterpret_cast<uint8_t*>(codes);
    const int64_t esz = dtype == 1 ? 2 : 4;
    if (axis == 1) {
        const Div32 dgl = make_div32((uint32_t)(cols / 8));
        const int64_t nchunks = rows * (cols / 8);
        if (dtype == 1)   // bf16: two chunks per thread at every size, as curvefp_quantize
            return launch_rows_u<F, true, 2>(src, rows, cols, ld, fidx, cp, scales, (int)cols, -1, dgl, s);
        if (nchunks >= (int64_t)2048 * 256 * 2)
            return launch_rows_u<F, false, 2>(src, rows, cols, ld, fidx, cp, scales, (int)cols, -1, dgl, s);
        return launch_rows_u<F, false, 1>(src, rows, cols, ld, fidx, cp, scales, (int)cols, -1, dgl, s);
    }
    const Div32 dgq = make_div32((uint32_t)(rows / 32));
    const bool tiled = rows % TT_ROWS == 0 && cols % 8 == 0 && (reinterpret_cast<uintptr_t>(src) & 15) == 0 &&
                       (ld * esz) % 16 == 0 && rows / TT_ROWS <= 65535;
    if (tiled) {
        const dim3 grid((unsigned)((cols + TT_COLS - 1) / TT_COLS), (unsigned)(rows / TT_ROWS));
        if (dtype == 1)
            hipLaunchKernelGGL((quantize_cols_tiled_kernel<F, true>), grid, dim3(256), 0, s, src, rows, cols, ld, cp,
                               scales, fidx, 1, (int64_t)1, dgq);
        else
            hipLaunchKernelGGL((quantize_cols_tiled_kernel<F, false>), grid, dim3(256), 0, s, src, rows, cols, ld, cp,
                               scales, fidx, 1, (int64_t)1, dgq);
        return hipGetLastError();
    }
    return launch_cols<F, 1>(src, dtype, rows, cols, ld, fidx, cp, scales, (int)rows, 1, s);
}

template <class F>
hipError_t launch_compact_fmt(const void* src, int dtype, int64_t rows, int64_t cols, int64_t ld, int block, int S,
                              int fidx, void* codes, int8_t* row_ref, uint8_t* offsets, hipStream_t s) {
    const int64_t ob = (cols / block * S + 7) / 8;
    uint8_t* cp = reinterpret_cast<uint8_t*>(codes);
    if (dtype == 1)
        hipLaunchKernelGGL((quantize_compact_kernel<F, true>), dim3((unsigned)rows), dim3(256), 0, s, src, cols, ld,
                           block, S, cp, row_ref, offsets, ob, fidx);
    else
        hipLaunchKernelGGL((quantize_compact_kernel<F, false>), dim3((unsigned)rows), dim3(256), 0, s, src, cols, ld,
                           block, S, cp, row_ref, offsets, ob, fidx);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------------------------
// Static-operand scales (Sec. 3.1: weights quantized once pick, among representable powers of two,
// the scale that minimizes the squared reconstruction error).  One thread per block (of 32 here; larger blocks below): the block is quantized at each
// candidate scale a_c + u (a_c ceil-absmax; u = 0, -1, .., -(candidates - 1), then 1 .. P - 1
// when the level pattern spans P > 1 octaves), each element reconstructed to fp32 exactly as the
// dequantizer does, and the squared error summed in fp64 in index order; the first candidate
// with the least error wins.  Offline work for weights, run once per tensor.

// fp32 bits -> the same value in fp64, exactly, without the fp32 denormal mode's say
__device__ __forceinline__ double f64_of_f32_bits(uint32_t b) {
    const uint32_t e = (b >> 23) & 0xFFu, m = b & 0x7FFFFFu;
    double v;
    if (e == 0) {
        v = (double)m * 0x1p-149;                    // exact: m < 2^23, a power-of-two scale
    } else {
        const uint64_t d = ((uint64_t)(e - 127 + 1023) << 52) | ((uint64_t)m << 29);
        v = __builtin_bit_cast(double, d);
    }
    return (b >> 31) ? -v : v;
}

// acc + d * d as two roundings (no fused multiply-add), so the sum is the same everywhere
__device__ __forceinline__ double add_square(double acc, double d) {
#pragma clang fp contract(off)
    const double sq = d * d;
    return acc + sq;
}

// rank of one magnitude at scale a (the fast or the exact path of ranks_of)
template <class F>
__device__ __forceinline__ uint32_t rank_at(uint32_t mag, int a, const uint32_t* lut) {
    return a >= F::A_FAST_MIN ? rank_fast<F>(mag, a, lut) : rank_exact<F>(mag, a, lut);
}

// squared reconstruction error of one element at scale a, added to acc (fp64, index order)
template <class F>
__device__ __forceinline__ double add_element_error(double acc, uint32_t m, uint32_t s, double x, int a,
                                                    const uint32_t* lut, const uint32_t* mant, const uint64_t* sig) {
    const uint32_t rk = rank_at<F>(m, a, lut);
    const uint32_t code = rk | ((rk != 0 ? s : 0u) << F::EC);
    const double xh = f64_of_f32_bits(value_bits<F>(code, a, mant, sig));
    return add_square(acc, x - xh);
}

// candidates per block at most: 8 below or at the ceil-absmax scale, P - 1 <= 2 above it
constexpr int MSE_MAXC = 10;

// One thread per block.  The block's magnitudes sit in LDS ([element][thread], so a wave's
// reads of one element are conflict-free); one pass over the 32 elements updates every
// candidate's error sum, each in index order, so each element is converted once and only the
// sums stay in registers (the candidate loop is unrolled and guarded by the wave-uniform count).
template <class F, bool BF16>
__global__ __launch_bounds__(256) void quantize_mse_kernel(
    const void* __restrict__ src, int64_t rows, int64_t cols, int64_t ld, int axis, int candidates,
    uint8_t* __restrict__ codes, int8_t* __restrict__ scales, int fidx) {
    __shared__ uint32_t lut[F::QLUT_SIZE];
    constexpr int RT = F::BINARY ? 8 : 128;
    __shared__ uint32_t mant[RT];
    __shared__ uint64_t sig[RT];
    __shared__ uint32_t smag[32 * 256];
    for (int i = threadIdx.x; i < F::QLUT_SIZE; i += blockDim.x) lut[i] = g_qlut[fidx][i];
    if (threadIdx.x < RT) {
        mant[threadIdx.x] = g_qr_mant[fidx][threadIdx.x];
        sig[threadIdx.x] = g_qr_sig[fidx][threadIdx.x];
    }
    const uint32_t lmax_mant = g_lmax_mant[fidx];
    __syncthreads();
    // block b: axis 1 -> row b / (cols / 32), block b mod (cols / 32) of it; axis 0 -> column
    // b mod cols, rows 32 (b / cols) ..: consecutive threads take consecutive columns
    const int64_t nbr = axis == 1 ? cols / 32 : rows / 32;          // blocks per output row
    const int64_t nb = axis == 1 ? rows * nbr : cols * nbr;
    const int64_t b = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (b >= nb) return;
    uint32_t* my = smag + threadIdx.x;                              // element i at my[256 i]
    int64_t orow, oblk;                                             // output row and block in it
    uint32_t sgn = 0, amax = 0;
    if (axis == 1) {
        orow = b / nbr;
        oblk = b - orow * nbr;
        if (BF16) {
            const uint4* p = reinterpret_cast<const uint4*>(reinterpret_cast<const uint16_t*>(src) + orow * ld + 32 * oblk);
#pragma unroll
            for (int t = 0; t < 4; t++) {
                const uint4 v = p[t];
                const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
                for (int j = 0; j < 4; j++) {
                    const uint32_t m0 = (w[j] << 16) & 0x7FFF0000u, m1 = w[j] & 0x7FFF0000u;
                    my[256 * (8 * t + 2 * j)] = m0;
                    my[256 * (8 * t + 2 * j + 1)] = m1;
                    amax = max(amax, max(m0, m1));
                    sgn |= ((w[j] >> 15) & 1u) << (8 * t + 2 * j);
                    sgn |= (w[j] >> 31) << (8 * t + 2 * j + 1);
                }
            }
        } else {
            const uint4* p = reinterpret_cast<const uint4*>(reinterpret_cast<const uint32_t*>(src) + orow * ld + 32 * oblk);
#pragma unroll
            for (int t = 0; t < 8; t++) {
                const uint4 v = p[t];
                const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
                for (int j = 0; j < 4; j++) {
                    const uint32_t m = w[j] & 0x7FFFFFFFu;
                    my[256 * (4 * t + j)] = m;
                    amax = max(amax, m);
                    sgn |= (w[j] >> 31) << (4 * t + j);
                }
            }
        }
    } else {
        const int64_t rb = b / cols;
        orow = b - rb * cols;                                       // the source column
        oblk = rb;
#pragma unroll
        for (int i = 0; i < 32; i++) {
            const int64_t e = (32 * rb + i) * ld + orow;
            const uint32_t w = BF16 ? ((uint32_t)reinterpret_cast<const uint16_t*>(src)[e] << 16)
                                    : reinterpret_cast<const uint32_t*>(src)[e];
            my[256 * i] = w & 0x7FFFFFFFu;
            amax = max(amax, w & 0x7FFFFFFFu);
            sgn |= (w >> 31) << i;
        }
    }
    const int ac = scale_of<F>(amax, lmax_mant);
    const bool live = ac != -128 && amax != 0;
    int best_a = ac;
    if (live) {
        const int nc = candidates + F::PERIOD - 1;
        int acand[MSE_MAXC];
        bool ok[MSE_MAXC];
        double acc[MSE_MAXC];
#pragma unroll
        for (int c = 0; c < MSE_MAXC; c++) {
            acand[c] = c < candidates ? ac - c : ac + (c - candidates + 1);
            ok[c] = c < nc && acand[c] >= -127 && acand[c] <= 127;
            acc[c] = 0.0;
        }
#pragma unroll 2
        for (int i = 0; i < 32; i++) {
            const uint32_t m = my[256 * i];
            const uint32_t s = (sgn >> i) & 1u;
            const double x = f64_of_f32_bits(m | (s << 31));
#pragma unroll
            for (int c = 0; c < MSE_MAXC; c++)
                if (c < nc && ok[c]) acc[c] = add_element_error<F>(acc[c], m, s, x, acand[c], lut, mant, sig);
        }
        // the first candidate in the order above with the least error
        double best_err = acc[0];
#pragma unroll
        for (int c = 1; c < MSE_MAXC; c++)
            if (c < nc && ok[c] && acc[c] < best_err) {
                best_err = acc[c];
                best_a = acand[c];
            }
    }
    uint32_t cc[32];
#pragma unroll
    for (int i = 0; i < 32; i++) {
        const uint32_t rk = live ? rank_at<F>(my[256 * i], best_a, lut) : 0u;
        cc[i] = rk | ((rk != 0 ? (sgn >> i) & 1u : 0u) << F::EC);
    }
    if (!F::PACKED7) {
        uint4* o = reinterpret_cast<uint4*>(codes + (orow * nbr + oblk) * 32);
#pragma unroll
        for (int q = 0; q < 2; q++) {
            uint32_t k[4];
#pragma unroll
            for (int j = 0; j < 4; j++)
                k[j] = cc[16 * q + 4 * j] | (cc[16 * q + 4 * j + 1] << 8) | (cc[16 * q + 4 * j + 2] << 16) |
                       (cc[16 * q + 4 * j + 3] << 24);
            o[q] = make_uint4(k[0], k[1], k[2], k[3]);
        }
    } else {
        uint32_t wds[7] = {0, 0, 0, 0, 0, 0, 0};
#pragma unroll
        for (int i = 0; i < 32; i++) {
            const int bit = 7 * i;
            wds[bit >> 5] |= cc[i] << (bit & 31);
            if ((bit & 31) > 25) wds[(bit >> 5) + 1] |= cc[i] >> (32 - (bit & 31));
        }
        uint32_t* o = reinterpret_cast<uint32_t*>(codes + (orow * nbr + oblk) * 28);
#pragma unroll
        for (int j = 0; j < 7; j++) o[j] = wds[j];
    }
    scales[orow * nbr + oblk] = (int8_t)best_a;
}

// The same search for blocks of G > 32 elements (Sec. 4.2's PTQ weights use G64 and G512): one
// thread per block streams it from memory three times (its maximum; every candidate's error
// sum, element by element in index order; the codes at the winning scale, 32 at a time), so
// only the candidates' sums stay in registers.  Blocks along rows are read 8 elements per
// 16-byte load; blocks down the columns one element per load (consecutive threads take
// consecutive columns).
template <class F, bool BF16>
__device__ __forceinline__ void mse_load8(const void* __restrict__ src, int axis, int64_t base, int64_t ld, int j,
                                          uint32_t* mag, uint32_t& sgn8) {
    sgn8 = 0;
    if (axis == 1) {
        const char* p = reinterpret_cast<const char*>(src) + (base + 8 * (int64_t)j) * (BF16 ? 2 : 4);
        uint4 v[BF16 ? 1 : 2];
#pragma unroll
        for (int t = 0; t < (BF16 ? 1 : 2); t++) v[t] = ld16<false>(reinterpret_cast<const uint4*>(p) + t);
        uint32_t sg[8];
        unpack8<BF16>(v, mag, sg);
#pragma unroll
        for (int e = 0; e < 8; e++) sgn8 |= sg[e] << e;
    } else {
#pragma unroll
        for (int e = 0; e < 8; e++) {
            const int64_t idx = base + (8 * (int64_t)j + e) * ld;
            const uint32_t w = BF16 ? ((uint32_t)reinterpret_cast<const uint16_t*>(src)[idx] << 16)
                                    : reinterpret_cast<const uint32_t*>(src)[idx];
            mag[e] = w & 0x7FFFFFFFu;
            sgn8 |= (w >> 31) << e;
        }
    }
}

template <class F, bool BF16>
__global__ __launch_bounds__(256) void quantize_mse_g_kernel(
    const void* __restrict__ src, int64_t rows, int64_t cols, int64_t ld, int axis, int G, int candidates,
    uint8_t* __restrict__ codes, int8_t* __restrict__ scales, int fidx) {
    __shared__ uint32_t lut[F::QLUT_SIZE];
    constexpr int RT = F::BINARY ? 8 : 128;
    __shared__ uint32_t mant[RT];
    __shared__ uint64_t sig[RT];
    for (int i = threadIdx.x; i < F::QLUT_SIZE; i += blockDim.x) lut[i] = g_qlut[fidx][i];
    if (threadIdx.x < RT) {
        mant[threadIdx.x] = g_qr_mant[fidx][threadIdx.x];
        sig[threadIdx.x] = g_qr_sig[fidx][threadIdx.x];
    }
    const uint32_t lmax_mant = g_lmax_mant[fidx];
    __syncthreads();
    const int64_t k = axis == 1 ? cols : rows;                   // blocked extent
    const int64_t nbr = k / G;                                    // blocks per output row
    const int64_t nb = axis == 1 ? rows * nbr : cols * nbr;
    const int64_t b = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (b >= nb) return;
    int64_t orow, oblk, base;                                     // output row, block, first element
    if (axis == 1) {
        orow = b / nbr;
        oblk = b - orow * nbr;
        base = orow * ld + oblk * G;
    } else {
        oblk = b / cols;
        orow = b - oblk * cols;                                   // the source column
        base = oblk * G * ld + orow;
    }
    const int nch = G / 8;
    uint32_t amax = 0;
    for (int j = 0; j < nch; j++) {
        uint32_t mag[8], sg;
        mse_load8<F, BF16>(src, axis, base, ld, j, mag, sg);
#pragma unroll
        for (int e = 0; e < 8; e++) amax = max(amax, mag[e]);
    }
    const int ac = scale_of<F>(amax, lmax_mant);
    const bool live = ac != -128 && amax != 0;
    int best_a = ac;
    if (live) {
        const int nc = candidates + F::PERIOD - 1;
        int acand[MSE_MAXC];
        bool ok[MSE_MAXC];
        double acc[MSE_MAXC];
#pragma unroll
        for (int c = 0; c < MSE_MAXC; c++) {
            acand[c] = c < candidates ? ac - c : ac + (c - candidates + 1);
            ok[c] = c < nc && acand[c] >= -127 && acand[c] <= 127;
            acc[c] = 0.0;
        }
        for (int j = 0; j < nch; j++) {
            uint32_t mag[8], sg;
            mse_load8<F, BF16>(src, axis, base, ld, j, mag, sg);
#pragma unroll
            for (int e = 0; e < 8; e++) {
                const uint32_t s = (sg >> e) & 1u;
                const double x = f64_of_f32_bits(mag[e] | (s << 31));
#pragma unroll
                for (int c = 0; c < MSE_MAXC; c++)
                    if (c < nc && ok[c])
                        acc[c] = add_element_error<F>(acc[c], mag[e], s, x, acand[c], lut, mant, sig);
            }
        }
        double best_err = acc[0];
#pragma unroll
        for (int c = 1; c < MSE_MAXC; c++)
            if (c < nc && ok[c] && acc[c] < best_err) {
                best_err = acc[c];
                best_a = acand[c];
            }
    }
    // codes, one group of 32 at a time
    for (int grp = 0; grp < G / 32; grp++) {
        uint32_t cc[32];
#pragma unroll
        for (int q = 0; q < 4; q++) {
            uint32_t mag[8], sg;
            mse_load8<F, BF16>(src, axis, base, ld, 4 * grp + q, mag, sg);
#pragma unroll
            for (int e = 0; e < 8; e++) {
                const uint32_t rk = live ? rank_at<F>(mag[e], best_a, lut) : 0u;
                cc[8 * q + e] = rk | ((rk != 0 ? (sg >> e) & 1u : 0u) << F::EC);
            }
        }
        const int64_t g32 = orow * (k / 32) + oblk * (G / 32) + grp;   // group of 32 in the output
        if (!F::PACKED7) {
            uint4* o = reinterpret_cast<uint4*>(codes + g32 * 32);
#pragma unroll
            for (int h = 0; h < 2; h++) {
                uint32_t w4[4];
#pragma unroll
                for (int t = 0; t < 4; t++)
                    w4[t] = cc[16 * h + 4 * t] | (cc[16 * h + 4 * t + 1] << 8) | (cc[16 * h + 4 * t + 2] << 16) |
                            (cc[16 * h + 4 * t + 3] << 24);
                o[h] = make_uint4(w4[0], w4[1], w4[2], w4[3]);
            }
        } else {
            uint32_t wds[7] = {0, 0, 0, 0, 0, 0, 0};
#pragma unroll
            for (int i = 0; i < 32; i++) {
                const int bit = 7 * i;
                wds[bit >> 5] |= cc[i] << (bit & 31);
                if ((bit & 31) > 25) wds[(bit >> 5) + 1] |= cc[i] >> (32 - (bit & 31));
            }
            uint32_t* o = reinterpret_cast<uint32_t*>(codes + g32 * 28);
#pragma unroll
            for (int t = 0; t < 7; t++) o[t] = wds[t];
        }
    }
    scales[orow * nbr + oblk] = (int8_t)best_a;
}

template <class F>
hipError_t launch_mse_fmt(const void* src, int dtype, int64_t rows, int64_t cols, int64_t ld, int axis,
                          int block, int candidates, int fidx, void* codes, int8_t* scales, hipStream_t s) {
    uint8_t* cp = reinterpret_cast<uint8_t*>(codes);
    if (block > 32) {
        const int64_t nbg = rows * cols / block;
        const dim3 gg((unsigned)((nbg + 255) / 256));
        if (dtype == 1)
            hipLaunchKernelGGL((quantize_mse_g_kernel<F, true>), gg, dim3(256), 0, s, src, rows, cols, ld, axis, block,
                               candidates, cp, scales, fidx);
        else
            hipLaunchKernelGGL((quantize_mse_g_kernel<F, false>), gg, dim3(256), 0, s, src, rows, cols, ld, axis, block,
                               candidates, cp, scales, fidx);
        return hipGetLastError();
    }
    const int64_t nb = rows * cols / 32;
    const dim3 grid((unsigned)((nb + 255) / 256));
    if (dtype == 1)
        hipLaunchKernelGGL((quantize_mse_kernel<F, true>), grid, dim3(256), 0, s, src, rows, cols, ld, axis, candidates,
                           cp, scales, fidx);
    else
        hipLaunchKernelGGL((quantize_mse_kernel<F, false>), grid, dim3(256), 0, s, src, rows, cols, ld, axis, candidates,
                           cp, scales, fidx);
    return hipGetLastError();
}


// ---------------------------------------------------------------------------------------------
// Quantize and prepare in one launch: Q(X) of Sec. 3.1 with blocks along the rows, then the
// result's staging as a GEMM operand (Sec. 3.3) -- the planes and row maxima that curvefp_prepare
// writes from these codes (planes.hpp) -- and, when dst is given, the reconstruction of
// Eq. curvefp-value that curvefp_dequantize writes.  WPR waves take one row (four rows per
// workgroup, or one), in two passes over its chunks (8 elements; in segment s, chunk
// g = 64 WPR (UL s + u) + 64 w + lane for wave w of the row, UL chunks per lane in flight): the
// first reads the source once, takes every block's scale and the row's largest scale key alpha
// (over the row's waves through LDS when WPR > 1) and keeps the chunks in LDS (64 WPR U per row,
// 32 KB per workgroup at most, so that several workgroups share a compute unit); the second
// takes them back and writes.  Slots past the row's end hold zeros (scale -127, the bottom key,
// so alpha is unchanged) and store nothing.  Workgroups of the padding rows (up to the next
// multiple of 256) write zero planes and a zero row maximum, as the expansion does past the
// operand.  Two operands of one GEMM (same k, format and source type) can share a launch:
// workgroups [0, blocks_a) take A, the rest B.
struct QPOperand {
    const void* src;
    int64_t rows, ld;
    uint8_t* codes;
    int8_t* scales;
    char* planes;
    int* rmax;          // the prepared layout's row maxima, after the planes
    int64_t RT;         // tiles of 256 rows
    float* dst;         // the reconstruction, or null
    int64_t ld_dst;
};

template <class F, bool BF16, int U, int WPR>
__global__ __launch_bounds__(256) void quantize_prepare_kernel(QPOperand opA, QPOperand opB, int64_t blocks_a,
                                                               uint32_t cpr, int64_t code_row_bytes, int64_t nsb,
                                                               int fidx, int lgl) {
    using T = typename std::conditional<BF16, uint8_t, uint32_t>::type;
    constexpr int ESZ = BF16 ? 2 : 4;
    constexpr int NV = BF16 ? 1 : 2;   // 16-byte loads per chunk
    constexpr int UL = U < 4 ? U : 4;
    constexpr uint32_t SPAN = 64u * WPR;   // chunks of a row per u step
    static_assert(WPR == 1 || WPR == 4, "one wave per row or one workgroup per row");
    static_assert(GEMM_DEC_ENTRIES == 256, "one expansion entry per thread");
    static_assert(4 * 64 * U * NV * 16 <= 32768, "LDS staging of at most 32 KB per workgroup");
    __shared__ __attribute__((aligned(16))) uint4 rowbuf[4 * 64 * U * NV];
    __shared__ __attribute__((aligned(16))) T lut[F::QLUT_SIZE];
    __shared__ uint32_t dec[GEMM_DEC_ENTRIES];
    __shared__ uint32_t qmant[128];
    __shared__ uint64_t qsig[128];
    __shared__ int wkey[4];
    const int lane = (int)(threadIdx.x & 63), wave = (int)(threadIdx.x >> 6);
    const bool isA = (int64_t)blockIdx.x < blocks_a;
    const QPOperand& op = isA ? opA : opB;
    const int64_t bid = isA ? (int64_t)blockIdx.x : (int64_t)blockIdx.x - blocks_a;
    const int64_t rows = op.rows, ld = op.ld, RT = op.RT, ld_dst = op.ld_dst;
    char* __restrict__ planes = op.planes;
    float* __restrict__ dst = op.dst;
    const int wr = wave % WPR;                               // this wave's part of its row
    const int64_t row = (bid * 4 + wave) / WPR;
    const bool real = row < rows;                            // uniform over the waves of a row
    uint4* wbuf = rowbuf + (wave / WPR) * (SPAN * U * NV);
    const uint4* srow = reinterpret_cast<const uint4*>(reinterpret_cast<const char*>(op.src) + (real ? row : 0) * ld * ESZ);
    const uint32_t nseg = (cpr + SPAN * UL - 1) / (SPAN * UL);
    auto chunk_of = [&](uint32_t seg, int u) { return SPAN * (UL * seg + (uint32_t)u) + 64u * wr + (uint32_t)lane; };
    auto load = [&](uint32_t seg, uint4 (*v)[NV]) {
#pragma unroll
        for (int u = 0; u < UL; u++) {
            const uint32_t g = chunk_of(seg, u);
#pragma unroll
            for (int t = 0; t < NV; t++) v[u][t] = make_uint4(0u, 0u, 0u, 0u);
            if (real && g < cpr) {
#pragma unroll
                for (int t = 0; t < NV; t++) v[u][t] = ld16<true>(srow + NV * g + t);
            }
        }
    };
    // the first segment is requested before the tables are filled, so both latencies overlap
    uint4 cur[UL][NV];
    load(0, cur);
    if (BF16) {
        const uint32_t* s32 = reinterpret_cast<const uint32_t*>(g_qlut8[fidx]);
        uint32_t* l32 = reinterpret_cast<uint32_t*>(lut);
        for (int i = threadIdx.x; i < F::QLUT_SIZE / 4; i += blockDim.x) l32[i] = s32[i];
    } else {
        for (int i = threadIdx.x; i < F::QLUT_SIZE; i += blockDim.x) lut[i] = (T)g_qlut[fidx][i];
    }
    dec[threadIdx.x] = g_qp_dec[fidx][threadIdx.x];
    if (dst != nullptr && threadIdx.x < 128) {
        qmant[threadIdx.x] = g_qr_mant[fidx][threadIdx.x];
        qsig[threadIdx.x] = g_qr_sig[fidx][threadIdx.x];
    }
    const uint32_t lmax_mant = g_lmax_mant[fidx];
    __syncthreads();

    const int64_t rt = row / BM;
    const int rr = (int)(row - rt * BM);
    if (!real) {   // the whole row's waves (and, for WPR = 4, the workgroup) leave here
        if (row < RT * BM) {
            for (uint32_t g = 64u * wr + (uint32_t)lane; g < cpr; g += SPAN) {
                char* pd = planes + ((int64_t)(g >> 2) * RT + rt) * (2 * PLANE) + swz(rr, (int)(g & 3));
                *reinterpret_cast<uint4*>(pd) = make_uint4(0u, 0u, 0u, 0u);
                *reinterpret_cast<uint4*>(pd + PLANE) = make_uint4(0u, 0u, 0u, 0u);
            }
            if (wr == 0 && lane == 0) op.rmax[row] = 0;
        }
        return;
    }

    // the block scale of a chunk: the 2^lgl lanes of a block share its largest magnitude
    auto chunk_scale = [&](const uint4* v) {
        uint32_t mag[8], sgn[8];
        unpack8<BF16>(v, mag, sgn);
        uint32_t amax = 0;
#pragma unroll
        for (int i = 0; i < 8; i++) amax = max(amax, mag[i]);
        amax = lgl == 2 ? quad_max_u32(amax) : group_max_u32(amax, lgl);
        return scale_of<F>(amax, lmax_mant);
    };

    // pass 1: the row's top key; the chunks go to LDS
    int key = -128;
    for (uint32_t seg = 0; seg < nseg; seg++) {
        uint4 nxt[UL][NV];
        if (seg + 1 < nseg) load(seg + 1, nxt);
#pragma unroll
        for (int u = 0; u < UL; u++) {
            key = max(key, scale_key(chunk_scale(cur[u])));
            const uint32_t g = chunk_of(seg, u);
#pragma unroll
            for (int t = 0; t < NV; t++) wbuf[NV * g + t] = cur[u][t];
        }
#pragma unroll
        for (int u = 0; u < UL; u++)
#pragma unroll
            for (int t = 0; t < NV; t++) cur[u][t] = nxt[u][t];
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) key = max(key, __shfl_xor(key, o));
    if (WPR > 1) {
        if (lane == 0) wkey[wave] = key;
        __syncthreads();
        key = max(max(wkey[0], wkey[1]), max(wkey[2], wkey[3]));
    }
    const int alpha = key;

    // pass 2: codes and scales, both planes, the reconstruction
    uint8_t* crow = op.codes + row * code_row_bytes;
    int8_t* scrow = op.scales + row * nsb;
    for (uint32_t seg = 0; seg < nseg; seg++) {
#pragma unroll
        for (int u = 0; u < UL; u++) {
            const uint32_t g = chunk_of(seg, u);
            uint4 v[NV];
#pragma unroll
            for (int t = 0; t < NV; t++) v[t] = wbuf[NV * g + t];
            const int a = chunk_scale(v);
            if (g >= cpr) continue;   // whole blocks: cpr is a multiple of a block's lanes
            uint32_t mag[8], sgn[8];
            unpack8<BF16>(v, mag, sgn);
            uint32_t c[8];
            chunk_codes<F>(mag, sgn, a, lut, c);
            store_codes<F, true>(c, g, crow);
            if ((g & ((1u << lgl) - 1)) == 0) scrow[g >> lgl] = (int8_t)a;
            uint32_t e[8];
#pragma unroll
            for (int i = 0; i < 8; i++) e[i] = dec[c[i]];
            uint32_t hv[4], lv[4];
            expand_chunk8(e, alpha - a, hv, lv);
            char* pd = planes + ((int64_t)(g >> 2) * RT + rt) * (2 * PLANE) + swz(rr, (int)(g & 3));
            *reinterpret_cast<uint4*>(pd) = make_uint4(hv[0], hv[1], hv[2], hv[3]);
            *reinterpret_cast<uint4*>(pd + PLANE) = make_uint4(lv[0], lv[1], lv[2], lv[3]);
            if (dst != nullptr) {
                uint32_t o[8];
#pragma unroll
                for (int i = 0; i < 8; i++) o[i] = a == -128 ? 0x7FC00000u : value_bits<F>(c[i], a, qmant, qsig);
                uint4* out = reinterpret_cast<uint4*>(dst + row * ld_dst + (int64_t)g * 8);
                out[0] = make_uint4(o[0], o[1], o[2], o[3]);
                out[1] = make_uint4(o[4], o[5], o[6], o[7]);
            }
        }
    }
    if (wr == 0 && lane == 0) op.rmax[row] = alpha;
}

// an operand of a launch: its buffers and tiles (rows = 0: none)
QPOperand qp_operand(const void* src, int64_t rows, int64_t k, int64_t ld, void* codes, int8_t* scales, void* prepared,
                     float* dst, int64_t ld_dst) {
    QPOperand o;
    o.src = src;
    o.rows = rows;
    o.ld = ld;
    o.codes = reinterpret_cast<uint8_t*>(codes);
    o.scales = scales;
    o.planes = reinterpret_cast<char*>(prepared);
    o.RT = (rows + BM - 1) / BM;
    // the prepared layout: planes, then the row maxima
    o.rmax = rows > 0 ? reinterpret_cast<int*>(o.planes + (k / 32) * o.RT * 2 * PLANE) : nullptr;
    o.dst = dst;
    o.ld_dst = ld_dst;
    return o;
}

template <class F, bool BF16, int U, int WPR>
hipError_t launch_qp_u(const QPOperand& a, const QPOperand& b, int64_t k, int fidx, int block, hipStream_t s) {
    int lgl = 0;
    while ((8 << lgl) < block) lgl++;
    const int64_t code_row_bytes = F::PACKED7 ? k / 32 * 28 : k;
    const int64_t blocks_a = a.RT * 64 * WPR, blocks_b = b.RT * 64 * WPR;
    hipLaunchKernelGGL((quantize_prepare_kernel<F, BF16, U, WPR>), dim3((unsigned)(blocks_a + blocks_b)), dim3(256), 0,
                       s, a, b, blocks_a, (uint32_t)(k / 8), code_row_bytes, k / block, fidx, lgl);
    return hipGetLastError();
}

// Rows of up to 512 chunks (bf16; 256 fp32: 2, 4 or 8 chunks per lane) take one wave each,
// rows of up to 1024 bf16 (512 fp32) chunks one workgroup each, staged in at most 32 KB of LDS
// per workgroup; qp_fused_rows decides which rows go here at all.
template <class F, bool BF16>
hipError_t launch_qp(const QPOperand& a, const QPOperand& b, int64_t k, int fidx, int block, hipStream_t s) {
    const int64_t cpr = k / 8;
    if (cpr <= 128) return launch_qp_u<F, BF16, 2, 1>(a, b, k, fidx, block, s);
    if (cpr <= 256) return launch_qp_u<F, BF16, 4, 1>(a, b, k, fidx, block, s);
    if constexpr (BF16) {
        if (cpr <= 512) return launch_qp_u<F, BF16, 8, 1>(a, b, k, fidx, block, s);
        if (cpr <= 1024) return launch_qp_u<F, BF16, 4, 4>(a, b, k, fidx, block, s);
        return launch_qp_u<F, BF16, 8, 4>(a, b, k, fidx, block, s);
    } else {
        return launch_qp_u<F, BF16, 2, 4>(a, b, k, fidx, block, s);
    }
}

template <class F>
hipError_t launch_qp_fmt(const QPOperand& a, const QPOperand& b, int dtype, int64_t k, int fidx, int block,
                         hipStream_t s) {
    return dtype == 1 ? launch_qp<F, true>(a, b, k, fidx, block, s) : launch_qp<F, false>(a, b, k, fidx, block, s);
}

// Which shapes take the fused kernel: rows of up to 1024 chunks (bf16; 512 fp32), and bf16 rows of
// up to 2048 chunks in tensors of at most 2^26 elements; the others run the quantize, expansion and
// reconstruction kernels in turn.  Measured on bf16 sources against those kernels in one call:
// 8192 x 8192 (a workgroup per row, 4 chunks per lane) 101 against 123 us; 4096 x 11008 and
// 4096 x 14336 (8 chunks per lane) 74.5 and 85.6 against 81.6 and 95.5 us, but 8192 x 14336
// 226 against 201 us.  (Rows staged in 96-128 KB of LDS per workgroup, or read twice from the L2
// by one wave, were 15-40% slower on those shapes.)
bool qp_fused_rows(int dtype, int64_t rows, int64_t k) {
    const int64_t cpr = k / 8;
    // the launch's work-items (up to 256 per row, the padding rows included) stay below 2^32
    if (rows >= ((int64_t)1 << 23)) return false;
    if (dtype != 1) return cpr <= 512;
    return cpr <= 1024 || (cpr <= 2048 && rows * k <= ((int64_t)1 << 26));
}
}  // namespace

hipError_t launch_quantize(const void* src, int dtype, int64_t rows, int64_t cols, int64_t ld,
                           int axis, int format, int block, void* codes, int8_t* scales, hipStream_t s) {
    switch (format) {
        case 0: return launch_fmt<FmtE4C3>(src, dtype, rows, cols, ld, axis, 0, block, codes, scales, s);
        case 1: return launch_fmt<FmtE5C2>(src, dtype, rows, cols, ld, axis, 1, block, codes, scales, s);
        case 2: return launch_fmt<FmtE3C3>(src, dtype, rows, cols, ld, axis, 2, block, codes, scales, s);
        case 3: return launch_fmt<FmtE4C3R89>(src, dtype, rows, cols, ld, axis, 3, block, codes, scales, s);
        default: return launch_fmt<FmtE4C3R34>(src, dtype, rows, cols, ld, axis, 4, block, codes, scales, s);
    }
}

}  // namespace curvefp

namespace curvefp {

namespace {

// the three kernels in turn for one operand (shapes the fused kernel does not take)
hipError_t qp_separate(const void* src, int dtype, int64_t rows, int64_t k, int64_t ld, int format, int block,
                       void* codes, int8_t* scales, void* prepared, float* dst, int64_t ld_dst, hipStream_t s) {
    hipError_t e = launch_quantize(src, dtype, rows, k, ld, 1, format, block, codes, scales, s);
    if (e == hipSuccess) e = launch_prepare(codes, scales, rows, k, format, block, 0, prepared, s);
    if (e == hipSuccess && dst != nullptr) e = launch_dequantize(codes, scales, format, rows, k, block, dst, ld_dst, s);
    return e;
}

hipError_t qp_launch(const QPOperand& a, const QPOperand& b, int dtype, int64_t k, int format, int block,
                     hipStream_t s) {
    switch (format) {
        case 0: return launch_qp_fmt<FmtE4C3>(a, b, dtype, k, 0, block, s);
        case 1: return launch_qp_fmt<FmtE5C2>(a, b, dtype, k, 1, block, s);
        case 2: return launch_qp_fmt<FmtE3C3>(a, b, dtype, k, 2, block, s);
        case 3: return launch_qp_fmt<FmtE4C3R89>(a, b, dtype, k, 3, block, s);
        default: return launch_qp_fmt<FmtE4C3R34>(a, b, dtype, k, 4, block, s);
    }
}

}  // namespace

hipError_t launch_quantize_prepare(const void* src, int dtype, int64_t rows, int64_t k, int64_t ld, int format,
                                  int block, void* codes, int8_t* scales, void* prepared, float* dst, int64_t ld_dst,
                                  hipStream_t s) {
    if (!qp_fused_rows(dtype, rows, k))
        return qp_separate(src, dtype, rows, k, ld, format, block, codes, scales, prepared, dst, ld_dst, s);
    const QPOperand none = qp_operand(nullptr, 0, k, 0, nullptr, nullptr, nullptr, nullptr, 0);
    return qp_launch(qp_operand(src, rows, k, ld, codes, scales, prepared, dst, ld_dst), none, dtype, k, format, block,
                     s);
}

hipError_t launch_quantize_prepare_pair(const void* src_a, int64_t rows_a, int64_t ld_a, void* codes_a,
                                       int8_t* scales_a, void* prepared_a, float* dst_a, int64_t ld_dst_a,
                                       const void* src_b, int64_t rows_b, int64_t ld_b, void* codes_b,
                                       int8_t* scales_b, void* prepared_b, float* dst_b, int64_t ld_dst_b, int dtype,
                                       int64_t k, int format, int block, hipStream_t s) {
    if (!qp_fused_rows(dtype, rows_a + rows_b, k)) {
        // too large together: each operand on its own (the fused kernel where it takes it alone)
        hipError_t e = launch_quantize_prepare(src_a, dtype, rows_a, k, ld_a, format, block, codes_a, scales_a,
                                               prepared_a, dst_a, ld_dst_a, s);
        if (e != hipSuccess) return e;
        return launch_quantize_prepare(src_b, dtype, rows_b, k, ld_b, format, block, codes_b, scales_b, prepared_b,
                                       dst_b, ld_dst_b, s);
    }
    return qp_launch(qp_operand(src_a, rows_a, k, ld_a, codes_a, scales_a, prepared_a, dst_a, ld_dst_a),
                     qp_operand(src_b, rows_b, k, ld_b, codes_b, scales_b, prepared_b, dst_b, ld_dst_b), dtype, k,
                     format, block, s);
}

hipError_t launch_quantize_mse(const void* src, int dtype, int64_t rows, int64_t cols, int64_t ld, int axis,
                               int format, int block, int candidates, void* codes, int8_t* scales, hipStream_t s) {
    switch (format) {
        case 0: return launch_mse_fmt<FmtE4C3>(src, dtype, rows, cols, ld, axis, block, candidates, 0, codes, scales, s);
        case 1: return launch_mse_fmt<FmtE5C2>(src, dtype, rows, cols, ld, axis, block, candidates, 1, codes, scales, s);
        case 2: return launch_mse_fmt<FmtE3C3>(src, dtype, rows, cols, ld, axis, block, candidates, 2, codes, scales, s);
        case 3: return launch_mse_fmt<FmtE4C3R89>(src, dtype, rows, cols, ld, axis, block, candidates, 3, codes, scales, s);
        default: return launch_mse_fmt<FmtE4C3R34>(src, dtype, rows, cols, ld, axis, block, candidates, 4, codes, scales, s);
    }
}

hipError_t launch_quantize_compact(const void* src, int dtype, int64_t rows, int64_t cols, int64_t ld, int format,
                                  int block, int scale_bits, void* codes, int8_t* row_ref, uint8_t* offsets,
                                  hipStream_t s) {
    switch (format) {
        case 0: return launch_compact_fmt<FmtE4C3>(src, dtype, rows, cols, ld, block, scale_bits, 0, codes, row_ref, offsets, s);
        case 1: return launch_compact_fmt<FmtE5C2>(src, dtype, rows, cols, ld, block, scale_bits, 1, codes, row_ref, offsets, s);
        case 2: return launch_compact_fmt<FmtE3C3>(src, dtype, rows, cols, ld, block, scale_bits, 2, codes, row_ref, offsets, s);
        case 3: return launch_compact_fmt<FmtE4C3R89>(src, dtype, rows, cols, ld, block, scale_bits, 3, codes, row_ref, offsets, s);
        default: return launch_compact_fmt<FmtE4C3R34>(src, dtype, rows, cols, ld, block, scale_bits, 4, codes, row_ref, offsets, s);
    }
}

hipError_t launch_scales_unpack(const int8_t* row_ref, const uint8_t* offsets, int64_t rows, int64_t nblocks,
                                int scale_bits, int8_t* scales, hipStream_t s) {
    const int64_t n = rows * nblocks;
    hipLaunchKernelGGL(scales_unpack_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, row_ref, offsets, rows,
                       nblocks, (nblocks * scale_bits + 7) / 8, scale_bits, scales);
    return hipGetLastError();
}

hipError_t launch_quantize_tensorwise(const void* src, int dtype, int64_t rows, int64_t cols, int64_t ld, int axis,
                                     int format, void* codes, int8_t* scales, void* workspace, hipStream_t s) {
    uint32_t* w = reinterpret_cast<uint32_t*>(workspace);
    switch (format) {
        case 0: return launch_tensorwise_fmt<FmtE4C3>(src, dtype, rows, cols, ld, axis, 0, codes, scales, w, s);
        case 1: return launch_tensorwise_fmt<FmtE5C2>(src, dtype, rows, cols, ld, axis, 1, codes, scales, w, s);
        case 2: return launch_tensorwise_fmt<FmtE3C3>(src, dtype, rows, cols, ld, axis, 2, codes, scales, w, s);
        case 3: return launch_tensorwise_fmt<FmtE4C3R89>(src, dtype, rows, cols, ld, axis, 3, codes, scales, w, s);
        default: return launch_tensorwise_fmt<FmtE4C3R34>(src, dtype, rows, cols, ld, axis, 4, codes, scales, w, s);
    }
}

}  // namespace curvefp
