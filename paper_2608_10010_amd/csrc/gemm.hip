// CurveFP GEMM on the gfx950 matrix cores.
//
// C[M][N] = deq(A)[M][K] . deq(B)[N][K]^T.  The paper forms every nonzero
// product in the code domain and sums the products phase by phase,
// sum_h 2^{h/H} N_h (Sec. 3.2, Eq. binned-accumulation).  Here the same sum is
// evaluated on MFMA: every code is expanded once per workgroup into an fp16
// pair (hi, lo) with hi + lo = 2^{x} 2^{k/K} to 22 significant bits, where the
// exponent x = (a_b - alpha_row) + e + bias carries the block scale relative to
// the largest block scale alpha_row of its row (a power of two, so no new
// phase).  Three f16 MFMA products hi.hi + hi.lo + lo.hi accumulate in fp32,
// and the epilogue multiplies by 2^{alpha_i + beta_j - 2 bias} exactly.
//
// Expansion: a 256-entry table (sign included) gives the pair for a block at
// its row's largest scale; a block D = alpha_row - a_b binades lower is then
// scaled by 2^-D with one packed fp16 multiply per pair (exact while the
// result stays normal, correctly rounded below; D > 24 takes a second
// multiply).  The table is replicated 16 times in LDS so the lanes of a wave
// gather from different banks.
//
// Tiling: BM x BN output tile (256 x 256 or 256 x 128) per 512-thread
// workgroup, eight waves of WM x WN (MFMA 32x32x16 tiles), K step 32 = one
// scale block.  Expansion work is split into tasks of 8 codes (one 16-byte
// chunk of one row's hi and lo planes), BM+BN rows x 4 chunks spread evenly
// over the 512 threads.  Expanded tiles are double-buffered in LDS; the codes
// are fetched from HBM two steps ahead.  In every step the waves on a SIMD
// run in opposite order -- one runs its MFMAs while the other expands the
// next step -- and one barrier closes the step.  Tile rows are 64 bytes with
// the four 16-byte chunks XOR-swizzled by ((row >> 1) ^ (row >> 3)) & 3, so
// fragment reads and expansion writes spread over the banks.
#include "curvefp_internal.hpp"

#include <cstring>

namespace curvefp {

__device__ uint32_t g_dec[3][GEMM_DEC_ENTRIES];

hipError_t gemm_upload(const AllTables& t) {
    uint32_t h[3][GEMM_DEC_ENTRIES];
    for (int f = 0; f < 3; f++) memcpy(h[f], t.f[f].dec, sizeof(h[f]));
    return hipMemcpyToSymbol(HIP_SYMBOL(g_dec), h, sizeof(h));
}

namespace {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef _Float16 half2v __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int BM = 256;
constexpr int BK = 32;
constexpr int NTHREADS = 512;
constexpr int LUT_COPIES = 16;
constexpr int LUT_BYTES = GEMM_DEC_ENTRIES * LUT_COPIES * 4;
constexpr int ROW_BYTES = BK * 2;          // one fp16 plane row: 32 halves

template <int BN>
struct Tile {
    static constexpr int WM = (BN == 256) ? 128 : 64;    // wave tile rows
    static constexpr int WN = 64;                          // wave tile cols
    static constexpr int WAVES_N = BN / WN;
    static constexpr int TM = WM / 32, TN = WN / 32;       // MFMA tiles per wave
    static constexpr int PLANE_A = BM * ROW_BYTES;         // bytes of one A plane (hi or lo)
    static constexpr int PLANE_B = BN * ROW_BYTES;
    static constexpr int STAGE = 2 * PLANE_A + 2 * PLANE_B;
    static constexpr int SMEM = LUT_BYTES + 2 * STAGE + (BM + BN) * 4;
    static constexpr int TASKS_A = BM / 128;               // expansion tasks per thread
    static constexpr int TASKS = (BM + BN) / 128;
    static_assert((BM / WM) * WAVES_N == 8, "eight waves");
    static_assert(SMEM <= 160 * 1024, "LDS");
};

// byte offset of 16-byte chunk q (k = 8q .. 8q+7) of tile row r
// (the row term ((r >> 1) ^ (r >> 3)) & 3 spreads 16 consecutive rows over 64 banks and
// 8 consecutive rows over 32 banks for the 16-byte fragment reads)
__device__ __forceinline__ int swz(int r, int q) { return r * ROW_BYTES + 16 * (q ^ (((r >> 1) ^ (r >> 3)) & 3)); }

__device__ __forceinline__ uint32_t f16_pow2_neg(int d) {
    // bits of the fp16 value 2^-d for 0 <= d <= 24 (subnormal below 2^-14)
    return d <= 14 ? (uint32_t)(15 - d) << 10 : 1u << (24 - d);
}

// raw codes of one 8-code chunk: 8-bit formats read 8 bytes; E3C3 reads the
// dwords that hold bytes [7q, 7q+7) of the block's 28 bytes and aligns the 56
// code bits to bit 0
template <class F>
struct Raw {
    uint32_t w[2];
    int a;
};

template <class F>
__device__ __forceinline__ void load_raw(const uint8_t* row_codes, int64_t kb, int q, const int8_t* row_scl,
                                         Raw<F>& r) {
    if (!F::PACKED7) {
        const uint2 v = *reinterpret_cast<const uint2*>(row_codes + kb * 32 + q * 8);
        r.w[0] = v.x;
        r.w[1] = v.y;
    } else {
        const uint32_t* p = reinterpret_cast<const uint32_t*>(row_codes + kb * 28);
        const int d0 = (7 * q) >> 2;
        const int sh = 8 * ((7 * q) & 3);
        const uint64_t lo = (uint64_t)p[d0] | ((uint64_t)p[d0 + 1] << 32);
        const uint64_t hi = sh > 8 ? (uint64_t)p[d0 + 2] : 0ull;
        const uint64_t v = sh ? ((lo >> sh) | (hi << (64 - sh))) : lo;
        r.w[0] = (uint32_t)v;
        r.w[1] = (uint32_t)(v >> 32);
    }
    r.a = row_scl[kb];
}

template <class F>
__device__ __forceinline__ uint32_t chunk_code(const Raw<F>& r, int i) {
    if (!F::PACKED7) return (r.w[i >> 2] >> (8 * (i & 3))) & 0xFFu;
    const uint64_t v = (uint64_t)r.w[0] | ((uint64_t)r.w[1] << 32);
    return (uint32_t)(v >> (7 * i)) & 0x7Fu;
}

template <class F>
__device__ __forceinline__ void expand_chunk(const Raw<F>& r, int alpha, const uint32_t* lut,
                                             int copy4, char* hi_dst, char* lo_dst) {
    uint32_t e[8];
#pragma unroll
    for (int i = 0; i < 8; i++) {
        const uint32_t c = chunk_code<F>(r, i);
        e[i] = *reinterpret_cast<const uint32_t*>(reinterpret_cast<const char*>(lut) + (c << 6) + copy4);
    }
    uint32_t hv[4], lv[4];
#pragma unroll
    for (int p = 0; p < 4; p++) {
        hv[p] = __builtin_amdgcn_perm(e[2 * p + 1], e[2 * p], 0x05040100u);
        lv[p] = __builtin_amdgcn_perm(e[2 * p + 1], e[2 * p], 0x07060302u);
    }
    const int D = alpha - r.a;      // >= 0
    if (D != 0) {
        const int d1 = D < 24 ? D : 24;
        const uint32_t s1 = f16_pow2_neg(d1) * 0x10001u;
        const half2v m1 = __builtin_bit_cast(half2v, s1);
#pragma unroll
        for (int p = 0; p < 4; p++) {
            hv[p] = __builtin_bit_cast(uint32_t, __builtin_bit_cast(half2v, hv[p]) * m1);
            lv[p] = __builtin_bit_cast(uint32_t, __builtin_bit_cast(half2v, lv[p]) * m1);
        }
        if (D > 24) {
            const int d2 = D - 24 < 24 ? D - 24 : 24;
            const half2v m2 = __builtin_bit_cast(half2v, f16_pow2_neg(d2) * 0x10001u);
#pragma unroll
            for (int p = 0; p < 4; p++) {
                hv[p] = __builtin_bit_cast(uint32_t, __builtin_bit_cast(half2v, hv[p]) * m2);
                lv[p] = __builtin_bit_cast(uint32_t, __builtin_bit_cast(half2v, lv[p]) * m2);
            }
        }
    }
    *reinterpret_cast<uint4*>(hi_dst) = make_uint4(hv[0], hv[1], hv[2], hv[3]);
    *reinterpret_cast<uint4*>(lo_dst) = make_uint4(lv[0], lv[1], lv[2], lv[3]);
}

template <class F, int BN>
struct Tasks {
    using T = Tile<BN>;
    const uint8_t* codes[T::TASKS];     // row base of this task's operand row (null if outside)
    const int8_t* scl[T::TASKS];
    int alpha[T::TASKS];
    int hi_off[T::TASKS], lo_off[T::TASKS];
};

template <class F, int BN>
__global__ __launch_bounds__(NTHREADS) void gemm_kernel(
    const uint8_t* __restrict__ A, const int8_t* __restrict__ As,
    const uint8_t* __restrict__ B, const int8_t* __restrict__ Bs,
    int64_t M, int64_t N, int64_t K, float* __restrict__ C, int64_t ldc, int fidx) {
    using T = Tile<BN>;
    extern __shared__ __attribute__((aligned(16))) char smem[];
    uint32_t* lut = reinterpret_cast<uint32_t*>(smem);
    char* stage0 = smem + LUT_BYTES;
    int* sAlpha = reinterpret_cast<int*>(smem + LUT_BYTES + 2 * T::STAGE);
    int* sBeta = sAlpha + BM;

    const int tid = threadIdx.x;
    for (int i = tid; i < GEMM_DEC_ENTRIES * LUT_COPIES; i += NTHREADS) lut[i] = g_dec[fidx][i / LUT_COPIES];

    const int64_t m0 = (int64_t)blockIdx.y * BM, n0 = (int64_t)blockIdx.x * BN;
    const int64_t nkb = K / 32;
    const int64_t code_row_bytes = F::PACKED7 ? nkb * 28 : K;

    // largest block scale of every A and B row of the tile
    if (tid < BM + BN) {
        const bool isA = tid < BM;
        const int lrow = isA ? tid : tid - BM;
        const int64_t grow = (isA ? m0 : n0) + lrow;
        int alpha = -128;
        if (grow < (isA ? M : N)) {
            const int8_t* s = (isA ? As : Bs) + grow * nkb;
            for (int64_t kb = 0; kb < nkb; kb++) alpha = max(alpha, (int)s[kb]);
        }
        (isA ? sAlpha : sBeta)[lrow] = alpha;
    }
    __syncthreads();

    // expansion tasks: rows (tid >> 2) + 128 j of A (j < TASKS_A) then of B; chunk q = tid & 3
    const int q = tid & 3;
    const int copy4 = (tid & (LUT_COPIES - 1)) * 4;
    Tasks<F, BN> tk;
#pragma unroll
    for (int j = 0; j < T::TASKS; j++) {
        const bool isA = j < T::TASKS_A;
        const int lrow = (tid >> 2) + 128 * (isA ? j : j - T::TASKS_A);
        const int64_t grow = (isA ? m0 : n0) + lrow;
        const bool valid = grow < (isA ? M : N);
        tk.codes[j] = valid ? (isA ? A : B) + grow * code_row_bytes : nullptr;
        tk.scl[j] = valid ? (isA ? As : Bs) + grow * nkb : nullptr;
        tk.alpha[j] = isA ? sAlpha[lrow] : sBeta[lrow];
        const int off = isA ? swz(lrow, q) : 2 * T::PLANE_A + swz(lrow, q);
        tk.hi_off[j] = off;
        tk.lo_off[j] = off + (isA ? T::PLANE_A : T::PLANE_B);
    }

    Raw<F> rawA[T::TASKS], rawB[T::TASKS];   // two register sets, indexed only at compile time
    auto fetch = [&](int64_t kb, Raw<F>* dst) {
#pragma unroll
        for (int j = 0; j < T::TASKS; j++)
            if (tk.codes[j]) load_raw<F>(tk.codes[j], kb, q, tk.scl[j], dst[j]);
    };
    auto expand = [&](const Raw<F>* src, char* stage) {
#pragma unroll
        for (int j = 0; j < T::TASKS; j++) {
            if (tk.codes[j]) {
                expand_chunk<F>(src[j], tk.alpha[j], lut, copy4, stage + tk.hi_off[j], stage + tk.lo_off[j]);
            } else {
                *reinterpret_cast<uint4*>(stage + tk.hi_off[j]) = make_uint4(0, 0, 0, 0);
                *reinterpret_cast<uint4*>(stage + tk.lo_off[j]) = make_uint4(0, 0, 0, 0);
            }
        }
    };

    char* stage1 = stage0 + T::STAGE;
    fetch(0, rawA);
    if (nkb > 1) fetch(1, rawB);
    expand(rawA, stage0);

    const int lane = tid & 63, wave = tid >> 6;
    const int wm = wave / T::WAVES_N, wn = wave % T::WAVES_N;
    const bool mfma_first = (wave & 4) == 0;   // the two waves of a SIMD take opposite orders
    f32x16 acc[T::TM][T::TN];
#pragma unroll
    for (int i = 0; i < T::TM; i++)
#pragma unroll
        for (int j = 0; j < T::TN; j++)
#pragma unroll
            for (int v = 0; v < 16; v++) acc[i][j][v] = 0.f;
    __syncthreads();

    auto mfma_step = [&](const char* st) {
        const char* sAh = st;
        const char* sAl = st + T::PLANE_A;
        const char* sBh = st + 2 * T::PLANE_A;
        const char* sBl = sBh + T::PLANE_B;
#pragma unroll
        for (int kq = 0; kq < 2; kq++) {
            const int qq = 2 * kq + (lane >> 5);
            half8 ah[T::TM], al[T::TM], bh[T::TN], bl[T::TN];
#pragma unroll
            for (int t = 0; t < T::TM; t++) {
                const int r = wm * T::WM + t * 32 + (lane & 31);
                ah[t] = *reinterpret_cast<const half8*>(sAh + swz(r, qq));
                al[t] = *reinterpret_cast<const half8*>(sAl + swz(r, qq));
            }
#pragma unroll
            for (int t = 0; t < T::TN; t++) {
                const int r = wn * T::WN + t * 32 + (lane & 31);
                bh[t] = *reinterpret_cast<const half8*>(sBh + swz(r, qq));
                bl[t] = *reinterpret_cast<const half8*>(sBl + swz(r, qq));
            }
#pragma unroll
            for (int i = 0; i < T::TM; i++)
#pragma unroll
                for (int j = 0; j < T::TN; j++) {
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(ah[i], bh[j], acc[i][j], 0, 0, 0);
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(ah[i], bl[j], acc[i][j], 0, 0, 0);
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(al[i], bh[j], acc[i][j], 0, 0, 0);
                }
        }
    };

    // one step: MFMAs on `cur` (step kb), expansion of step kb+1 from `ex` into `nxt`,
    // codes of step kb+2 fetched into `fx` (the set step kb was expanded from)
    auto step = [&](int64_t kb, const char* cur, char* nxt, Raw<F>* fx, const Raw<F>* ex) {
        const bool more = kb + 1 < nkb;
        if (kb + 2 < nkb) fetch(kb + 2, fx);
        if (mfma_first) {
            mfma_step(cur);
            if (more) expand(ex, nxt);
        } else {
            if (more) expand(ex, nxt);
            mfma_step(cur);
        }
        __syncthreads();
    };
    for (int64_t kb = 0; kb < nkb; kb += 2) {
        step(kb, stage0, stage1, rawA, rawB);
        if (kb + 1 < nkb) step(kb + 1, stage1, stage0, rawB, rawA);
    }

    // epilogue: D[i][j], j = lane % 32, i = 8 (v / 4) + 4 (lane / 32) + v % 4
#pragma unroll
    for (int ti = 0; ti < T::TM; ti++)
#pragma unroll
        for (int tj = 0; tj < T::TN; tj++) {
            const int lj = wn * T::WN + tj * 32 + (lane & 31);
            const int64_t gj = n0 + lj;
            const int beta = sBeta[lj];
#pragma unroll
            for (int v = 0; v < 16; v++) {
                const int li = wm * T::WM + ti * 32 + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
                const int64_t gi = m0 + li;
                if (gi < M && gj < N)
                    C[gi * ldc + gj] = __builtin_amdgcn_ldexpf(acc[ti][tj][v], sAlpha[li] + beta - 2 * F::GEMM_BIAS);
            }
        }
}

template <class F, int BN>
hipError_t launch_tile(const void* a, const int8_t* as, const void* b, const int8_t* bs, int64_t M,
                       int64_t N, int64_t K, float* c, int64_t ldc, int fidx, hipStream_t s) {
    using T = Tile<BN>;
    // the dynamic-LDS limit is a per-function, per-device attribute: raise it once per device
    static bool attr_set[64] = {};
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
    if (!attr_set[dev]) {
        e = hipFuncSetAttribute(reinterpret_cast<const void*>(&gemm_kernel<F, BN>),
                                hipFuncAttributeMaxDynamicSharedMemorySize, T::SMEM);
        if (e != hipSuccess) return e;
        attr_set[dev] = true;
    }
    dim3 grid((unsigned)((N + BN - 1) / BN), (unsigned)((M + BM - 1) / BM));
    hipLaunchKernelGGL((gemm_kernel<F, BN>), grid, dim3(NTHREADS), T::SMEM, s,
                       reinterpret_cast<const uint8_t*>(a), as, reinterpret_cast<const uint8_t*>(b), bs,
                       M, N, K, c, ldc, fidx);
    return hipGetLastError();
}

template <class F>
hipError_t launch_fmt(const void* a, const int8_t* as, const void* b, const int8_t* bs, int64_t M,
                      int64_t N, int64_t K, float* c, int64_t ldc, int fidx, hipStream_t s) {
    // 256 x 256 tiles when they fill the 256 compute units at least twice, else 256 x 128
    const int64_t tiles256 = ((M + BM - 1) / BM) * ((N + 255) / 256);
    if (tiles256 >= 512)
        return launch_tile<F, 256>(a, as, b, bs, M, N, K, c, ldc, fidx, s);
    return launch_tile<F, 128>(a, as, b, bs, M, N, K, c, ldc, fidx, s);
}

}  // namespace

hipError_t launch_gemm(const void* a, const int8_t* as, const void* b, const int8_t* bs, int64_t M,
                       int64_t N, int64_t K, int format, float* c, int64_t ldc, hipStream_t s) {
    switch (format) {
        case 0: return launch_fmt<FmtE4C3>(a, as, b, bs, M, N, K, c, ldc, 0, s);
        case 1: return launch_fmt<FmtE5C2>(a, as, b, bs, M, N, K, c, ldc, 1, s);
        default: return launch_fmt<FmtE3C3>(a, as, b, bs, M, N, K, c, ldc, 2, s);
    }
}

}  // namespace curvefp
