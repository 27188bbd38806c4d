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
// The (hi, lo) pair of every magnitude rank at every scale offset D =
// alpha_row - a_b comes from a host-built table (rows D > 40 are zero: such
// elements lie below 2^-25 of their row's largest element in fp16 terms).
//
// Tiling (this version): 128 x 128 output tile per 256-thread workgroup, four
// waves of 64 x 64 (2 x 2 MFMA 32x32x16 tiles each), K step 32 (one scale block).
#include "curvefp_internal.hpp"

#include <cstring>

namespace curvefp {

__device__ uint32_t g_dec[3][GEMM_DROWS * 128];

hipError_t gemm_upload(const AllTables& t) {
    static uint32_t h[3][GEMM_DROWS * 128];
    for (int f = 0; f < 3; f++) memcpy(h[f], t.f[f].dec, sizeof(h[f]));
    return hipMemcpyToSymbol(HIP_SYMBOL(g_dec), h, sizeof(h));
}

namespace {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int BM = 128, BN = 128, BK = 32;
constexpr int LDS_STRIDE = BK + 8;   // fp16 elements per row, padded against bank conflicts

template <class F>
__device__ __forceinline__ void load_codes(const uint8_t* codes, int64_t row, int64_t K, int64_t kb,
                                           uint32_t* c /*32*/) {
    if (!F::PACKED7) {
        const uint4* p = reinterpret_cast<const uint4*>(codes + row * K + kb * 32);
        const uint4 v0 = p[0], v1 = p[1];
        const uint32_t w[8] = {v0.x, v0.y, v0.z, v0.w, v1.x, v1.y, v1.z, v1.w};
#pragma unroll
        for (int i = 0; i < 32; i++) c[i] = (w[i >> 2] >> (8 * (i & 3))) & 0xFFu;
    } else {
        const uint32_t* p = reinterpret_cast<const uint32_t*>(codes + (row * (K / 32) + kb) * 28);
        uint32_t w[8];
#pragma unroll
        for (int d = 0; d < 7; d++) w[d] = p[d];
        w[7] = 0;
#pragma unroll
        for (int i = 0; i < 32; i++) {
            const int bit = 7 * i, d = bit >> 5, s = bit & 31;
            uint32_t v = w[d] >> s;
            if (s > 25) v |= w[d + 1] << (32 - s);
            c[i] = v & 0x7Fu;
        }
    }
}

template <class F>
__global__ __launch_bounds__(256) void gemm_kernel(
    const uint8_t* __restrict__ A, const int8_t* __restrict__ As,
    const uint8_t* __restrict__ B, const int8_t* __restrict__ Bs,
    int64_t M, int64_t N, int64_t K, float* __restrict__ C, int64_t ldc, int fidx) {
    __shared__ uint32_t dec[GEMM_DROWS * 128];
    __shared__ _Float16 sAh[BM * LDS_STRIDE], sAl[BM * LDS_STRIDE];
    __shared__ _Float16 sBh[BN * LDS_STRIDE], sBl[BN * LDS_STRIDE];
    __shared__ int sAlpha[BM], sBeta[BN];

    const int tid = threadIdx.x;
    for (int i = tid; i < GEMM_DROWS * 128; i += 256) dec[i] = g_dec[fidx][i];

    const int64_t m0 = (int64_t)blockIdx.y * BM, n0 = (int64_t)blockIdx.x * BN;
    const int64_t nkb = K / 32;

    // thread -> one operand row: tid < 128 loads A row m0+tid, else B row n0+tid-128
    const bool isA = tid < 128;
    const int lrow = isA ? tid : tid - 128;
    const int64_t grow = isA ? m0 + lrow : n0 + lrow;
    const bool valid = grow < (isA ? M : N);
    const uint8_t* codes = isA ? A : B;
    const int8_t* scl = (isA ? As : Bs) + (valid ? grow : 0) * nkb;

    int alpha = -128;
    if (valid)
        for (int64_t kb = 0; kb < nkb; kb++) alpha = max(alpha, (int)scl[kb]);
    (isA ? sAlpha : sBeta)[lrow] = alpha;
    _Float16* dh = (isA ? sAh : sBh) + lrow * LDS_STRIDE;
    _Float16* dl = (isA ? sAl : sBl) + lrow * LDS_STRIDE;

    const int lane = tid & 63, wave = tid >> 6;
    const int wr = wave >> 1, wc = wave & 1;
    f32x16 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; i++)
#pragma unroll
        for (int j = 0; j < 2; j++)
#pragma unroll
            for (int v = 0; v < 16; v++) acc[i][j][v] = 0.f;

    __syncthreads();

    for (int64_t kb = 0; kb < nkb; kb++) {
        // decode this row's 32 codes of block kb into the LDS tile
        uint32_t hv[16], lv[16];
        if (valid) {
            uint32_t c[32];
            load_codes<F>(codes, grow, K, kb, c);
            const int D = min(alpha - (int)scl[kb], GEMM_DMAX + 1);
            const uint32_t* drow = dec + D * 128;
#pragma unroll
            for (int i = 0; i < 32; i += 2) {
                uint32_t e0 = drow[c[i] & F::MAG_MASK];
                uint32_t e1 = drow[c[i + 1] & F::MAG_MASK];
                e0 ^= ((c[i] >> F::EC) & 1u) * 0x80008000u;
                e1 ^= ((c[i + 1] >> F::EC) & 1u) * 0x80008000u;
                hv[i >> 1] = (e0 & 0xFFFFu) | (e1 << 16);
                lv[i >> 1] = (e0 >> 16) | (e1 & 0xFFFF0000u);
            }
        } else {
#pragma unroll
            for (int i = 0; i < 16; i++) hv[i] = lv[i] = 0;
        }
#pragma unroll
        for (int q = 0; q < 4; q++) {
            reinterpret_cast<uint4*>(dh)[q] = make_uint4(hv[4 * q], hv[4 * q + 1], hv[4 * q + 2], hv[4 * q + 3]);
            reinterpret_cast<uint4*>(dl)[q] = make_uint4(lv[4 * q], lv[4 * q + 1], lv[4 * q + 2], lv[4 * q + 3]);
        }
        __syncthreads();

#pragma unroll
        for (int kk = 0; kk < BK; kk += 16) {
            const int koff = kk + (lane >> 5) * 8;
            half8 ah[2], al[2], bh[2], bl[2];
#pragma unroll
            for (int t = 0; t < 2; t++) {
                const int ar = wr * 64 + t * 32 + (lane & 31);
                const int br = wc * 64 + t * 32 + (lane & 31);
                ah[t] = *reinterpret_cast<const half8*>(sAh + ar * LDS_STRIDE + koff);
                al[t] = *reinterpret_cast<const half8*>(sAl + ar * LDS_STRIDE + koff);
                bh[t] = *reinterpret_cast<const half8*>(sBh + br * LDS_STRIDE + koff);
                bl[t] = *reinterpret_cast<const half8*>(sBl + br * LDS_STRIDE + koff);
            }
#pragma unroll
            for (int i = 0; i < 2; i++)
#pragma unroll
                for (int j = 0; j < 2; j++) {
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(ah[i], bh[j], acc[i][j], 0, 0, 0);
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(ah[i], bl[j], acc[i][j], 0, 0, 0);
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(al[i], bh[j], acc[i][j], 0, 0, 0);
                }
        }
        __syncthreads();
    }

    // epilogue: D[i][j], j = lane % 32, i = 8 (v / 4) + 4 (lane / 32) + v % 4
#pragma unroll
    for (int ti = 0; ti < 2; ti++)
#pragma unroll
        for (int tj = 0; tj < 2; tj++) {
            const int lj = wc * 64 + tj * 32 + (lane & 31);
            const int64_t gj = n0 + lj;
            if (gj >= N) continue;
            const int beta = sBeta[lj];
#pragma unroll
            for (int v = 0; v < 16; v++) {
                const int li = wr * 64 + ti * 32 + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
                const int64_t gi = m0 + li;
                if (gi >= M) continue;
                const int sh = sAlpha[li] + beta - 2 * F::GEMM_BIAS;
                C[gi * ldc + gj] = __builtin_amdgcn_ldexpf(acc[ti][tj][v], sh);
            }
        }
}

template <class F>
hipError_t launch_fmt(const void* a, const int8_t* as, const void* b, const int8_t* bs, int64_t M,
                      int64_t N, int64_t K, float* c, int64_t ldc, int fidx, hipStream_t s) {
    dim3 grid((unsigned)((N + BN - 1) / BN), (unsigned)((M + BM - 1) / BM));
    hipLaunchKernelGGL((gemm_kernel<F>), grid, dim3(256), 0, s,
                       reinterpret_cast<const uint8_t*>(a), as, reinterpret_cast<const uint8_t*>(b), bs,
                       M, N, K, c, ldc, fidx);
    return hipGetLastError();
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
