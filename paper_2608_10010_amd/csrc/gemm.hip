// CurveFP GEMM on the gfx950 matrix cores.
//
// C[M][N] = deq(A)[M][K] . deq(B)[N][K]^T.  The paper forms every nonzero
// product in the code domain and sums the products phase by phase,
// sum_h 2^{h/H} N_h (Sec. 3.2, Eq. binned-accumulation).  Here the same sum is
// evaluated on MFMA: every code is expanded once per workgroup into an fp16
// pair (hi, lo) with hi + lo = 2^{x} 2^{f/N} to 22 significant bits (the level
// r^{n/K} = 2^{w + f/N}; binary radix: w = e, f/N = k/K), where the
// exponent x = (a_b - alpha_row) + w + bias carries the block scale relative to
// the largest block scale alpha_row of its row (a power of two, so no new
// phase).  Three f16 MFMA products hi.hi + hi.lo + lo.hi accumulate in fp32,
// and the epilogue multiplies by 2^{alpha_i + beta_j - 2 bias} exactly.
//
// Expansion: a 256-entry table (sign included) gives the pair for a block at
// its row's largest scale; a block D = alpha_row - a_b binades lower is then
// scaled by 2^-min(D, 24) with one packed fp16 multiply per pair (exact while
// the result stays normal, correctly rounded below).  Blocks with D > 24 get a
// second multiply in a separate pass before the step's barrier (rare: only
// rows whose block scales spread over more than 24 binades).  The table is
// replicated 16 times in LDS so the lanes of a wave gather from 16 banks.
//
// Tiling: 256 x 256 output tile per 256-thread workgroup, four waves of
// 128 x 128 (4 x 4 MFMA 32x32x16 tiles), K step 32 = one scale block.  The
// expansion of step kb+1 (8 tasks of 8 codes per thread: one 16-byte chunk of
// one row's hi and lo planes) is interleaved with the 96 MFMAs of step kb;
// operand fragments are double-buffered in registers and the codes are
// fetched from HBM two steps ahead, so the matrix pipe, the VALU, LDS and HBM
// work at the same time.  Expanded tiles are double-buffered in LDS with one
// barrier per step.  Tile rows are 64 bytes with the four 16-byte chunks
// XOR-swizzled by ((row >> 1) ^ (row >> 3)) & 3, so fragment reads and
// expansion writes spread over the banks.
//
// Small problems split K in two (grid.z = 2) so the grid covers the 256
// compute units; the two partial sums land in C through fp32 atomic adds on
// a zero-filled C, which is order-independent for two terms.
#include "codec.hpp"
#include "curvefp_internal.hpp"
#include "device_util.hpp"
#include "planes.hpp"
#include "curvefp_tables.inc"

#include <cstring>
#include <type_traits>

namespace curvefp {

// compile-time tables (curvefp_tables.inc, written at build time by gen_tables)
__constant__ uint32_t g_dec[NUM_FORMATS][GEMM_DEC_ENTRIES] = CURVEFP_DEC_INIT;
// output requantization: the quantize tables of every format (the quantizer's, quantize.hip)
__constant__ uint32_t g_gq_lut[NUM_FORMATS][QLUT_MAX] = CURVEFP_QLUT_INIT;

// the output quantizer's rule per format, for the launch
constexpr uint32_t kLmaxMant[NUM_FORMATS] = CURVEFP_LMAX_MANT_INIT;
constexpr int kQlutSize[NUM_FORMATS] = CURVEFP_QLUT_SIZE_INIT;
constexpr int kOz[NUM_FORMATS] = {FmtE4C3::OZ, FmtE5C2::OZ, FmtE3C3::OZ, FmtE4C3R89::OZ, FmtE4C3R34::OZ};
constexpr int kOhi[NUM_FORMATS] = {FmtE4C3::OHI, FmtE5C2::OHI, FmtE3C3::OHI, FmtE4C3R89::OHI, FmtE4C3R34::OHI};
constexpr int kEc[NUM_FORMATS] = {FmtE4C3::EC, FmtE5C2::EC, FmtE3C3::EC, FmtE4C3R89::EC, FmtE4C3R34::EC};
constexpr bool qlut_sizes_ok() {
    for (int f = 0; f < NUM_FORMATS; f++)
        if (kQlutSize[f] != (kOhi[f] - kOz[f] + 1) * 128) return false;
    return true;
}
static_assert(qlut_sizes_ok(), "generated quantizer tables match the formats' octave ranges");
constexpr QRule qrule(int f) { return QRule{kOz[f], kOhi[f], kQlutSize[f], kEc[f], kLmaxMant[f]}; }

namespace {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int NTHREADS = 256;
constexpr int WM = 128, TM = 4;
constexpr int LUT_COPIES = 16;
constexpr int LUT_BYTES = GEMM_DEC_ENTRIES * LUT_COPIES * 4;

// tile shape: 256 x BN_ outputs, four waves of 128 x BN_/2 (BN_ = 256 or 128)
template <int BN_>
struct Tile {
    static constexpr int BN = BN_;
    static constexpr int WN = BN / 2, TN = WN / 32;
    static constexpr int PLANE_B = BN * ROW_BYTES;
    static constexpr int STAGE = 2 * PLANE + 2 * PLANE_B;     // Ahi, Alo, Bhi, Blo
    static constexpr int SMEM = LUT_BYTES + 2 * STAGE + (BM + BN) * 4;
    static constexpr int TASKS_B = BN / 64;                    // B rows r0 + 64 j
    static constexpr int TASKS = 4 + TASKS_B;                  // expansion tasks per thread per step
    static constexpr int MFMA_PER_SUB = TM * TN * 3;           // per 16-wide k slice
    static constexpr int MFMA_PER_GROUP = 2 * MFMA_PER_SUB / TASKS;
    static_assert(SMEM <= 160 * 1024, "LDS budget");
    static_assert(2 * MFMA_PER_SUB == MFMA_PER_GROUP * TASKS && MFMA_PER_SUB % MFMA_PER_GROUP == 0,
                  "groups split the slices evenly");
};

// sched_group_barrier masks
constexpr int SG_VALU = 0x002, SG_MFMA = 0x008, SG_DS_RD = 0x100;

// the epilogue's NaN for an output whose row or column holds a poisoned block (row maxima at or
// above POISON_KEY): C = deq(A) deq(B)^T with the poisoned blocks reconstructing to NaN
__device__ __forceinline__ float poisoned(float v, int row_max, int col_max) {
    return (row_max >= POISON_KEY || col_max >= POISON_KEY) ? __builtin_nanf("") : v;
}

template <class F>
struct Raw {
    uint32_t w[F::PACKED7 ? 3 : 2];   // the loaded code dwords, not yet unpacked
    uint32_t a;                       // the aligned scale dword that holds the block scale byte
};

// a task's 8 codes (E3C3: 56 bits aligned to bit 0) and its block scale
struct Chunk {
    uint32_t w[2];
    int a;
};

typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// one task's codes and scale; codes/scales are buffer descriptors over this tile's rows,
// so rows past the matrix edge read as zero codes
template <class F>
__device__ __forceinline__ void load_raw(__amdgpu_buffer_rsrc_t codes, __amdgpu_buffer_rsrc_t scl,
                                         int voff_code, int soff_code, int voff_scl, int soff_scl, int q,
                                         Raw<F>& r) {
    if (!F::PACKED7) {
        const u32x2 v = __builtin_amdgcn_raw_buffer_load_b64(codes, voff_code, soff_code, 0);
        r.w[0] = v.x;
        r.w[1] = v.y;
    } else {
        // bytes [7q, 7q + 7) of the block's 28 bytes: voff_code points at dword (7q) >> 2
        r.w[0] = __builtin_amdgcn_raw_buffer_load_b32(codes, voff_code, soff_code, 0);
        r.w[1] = __builtin_amdgcn_raw_buffer_load_b32(codes, voff_code + 4, soff_code, 0);
        r.w[2] = __builtin_amdgcn_raw_buffer_load_b32(codes, voff_code + 8, soff_code, 0);
    }
    r.a = __builtin_amdgcn_raw_buffer_load_b32(scl, voff_scl, soff_scl, 0);
}

// unpack a task at the step that expands it.  The empty asm makes the loaded words opaque, so
// the compiler cannot pull the unpacking up to the loads, which sit two steps earlier: that
// would make each step wait for the codes it has just started to fetch.
template <class F>
__device__ __forceinline__ Chunk settle(Raw<F> r, int q, int ash) {
    Chunk c;
    if (!F::PACKED7) {
        asm volatile("" : "+v"(r.w[0]), "+v"(r.w[1]), "+v"(r.a));
        c.w[0] = r.w[0];
        c.w[1] = r.w[1];
    } else {
        asm volatile("" : "+v"(r.w[0]), "+v"(r.w[1]), "+v"(r.w[2]), "+v"(r.a));
        // bytes [7q, 7q + 7) of the block's 28: the dwords start at byte 4 floor(7q / 4)
        const int sh = 8 * ((7 * q) & 3);
        const uint64_t lo = (uint64_t)r.w[0] | ((uint64_t)r.w[1] << 32);
        const uint64_t v = sh ? ((lo >> sh) | ((uint64_t)r.w[2] << (64 - sh))) : lo;
        c.w[0] = (uint32_t)v;
        c.w[1] = (uint32_t)(v >> 32);
    }
    c.a = (int)__builtin_amdgcn_sbfe(r.a, ash, 8);
    return c;
}

template <class F>
__device__ __forceinline__ uint32_t chunk_code(const Chunk& r, int i) {
    if (!F::PACKED7) return (r.w[i >> 2] >> (8 * (i & 3))) & 0xFFu;
    const uint64_t v = (uint64_t)r.w[0] | ((uint64_t)r.w[1] << 32);
    return (uint32_t)(v >> (7 * i)) & 0x7Fu;
}

// expansion of one task, in two parts so the table gathers of the next task can be in flight
// while this one is packed: gather -> 8 table entries (lo16 << 16 | hi16)
template <class F>
__device__ __forceinline__ void gather_chunk(const Chunk& r, const char* lut, int copy4, uint32_t* e) {
#pragma unroll
    for (int i = 0; i < 8; i++) {
        const uint32_t c = chunk_code<F>(r, i);
        e[i] = *reinterpret_cast<const uint32_t*>(lut + (c << 6) + copy4);
    }
}

// pack the 8 entries into hi/lo pairs, scale by 2^-min(D, 24), store 16 B to each plane
__device__ __forceinline__ void finish_chunk(const uint32_t* e, int D, char* hi_dst, char* lo_dst) {
    const half2v m1 = __builtin_bit_cast(half2v, f16_pow2_neg(min(max(D, 0), 24)) * 0x10001u);
    uint32_t hv[4], lv[4];
#pragma unroll
    for (int p = 0; p < 4; p++) {
        hv[p] = pk_mul(__builtin_amdgcn_perm(e[2 * p + 1], e[2 * p], 0x05040100u), m1);
        lv[p] = pk_mul(__builtin_amdgcn_perm(e[2 * p + 1], e[2 * p], 0x07060302u), m1);
    }
    *reinterpret_cast<uint4*>(hi_dst) = make_uint4(hv[0], hv[1], hv[2], hv[3]);
    *reinterpret_cast<uint4*>(lo_dst) = make_uint4(lv[0], lv[1], lv[2], lv[3]);
}

// second scaling for a chunk whose block lies more than 24 binades below its row's top
__device__ __forceinline__ void rescale_chunk(char* dst, int D) {
    const int d2 = min(D - 24, 24);
    const half2v m2 = __builtin_bit_cast(half2v, f16_pow2_neg(d2) * 0x10001u);
    uint4 v = *reinterpret_cast<uint4*>(dst);
    v.x = pk_mul(v.x, m2);
    v.y = pk_mul(v.y, m2);
    v.z = pk_mul(v.z, m2);
    v.w = pk_mul(v.w, m2);
    *reinterpret_cast<uint4*>(dst) = v;
}

// cache policy of buffer accesses that must be coherent across the XCDs' L2 caches (sc1:
// device scope): stores reach the device's point of coherence before they count as done,
// and loads do not hit lines another XCD may hold stale
constexpr int AUX_DEVICE_COHERENT = 16;

template <int TN>
struct Frag {
    half8 ah[TM], al[TM], bh[TN], bl[TN];
};

// epilogue of a 256 x BN_ tile: D[i][j] of MFMA tile (ti, tj) is register v of lane l with
// j = l % 32 and i = 8 (v / 4) + 4 (l / 32) + v % 4; C = ldexp(D, alpha_i + beta_j - BIAS2)
// (exact; BIAS2 = bias_A + bias_B, the fp16 exponent offsets of the two operands' expansions),
// stored, or added with fp32 atomics when K is split
// (ADD: each value is added to the other K half's value of the same element, read from its
// partial-tile slot at `other`, at wbase in the layout the workspace kernel writes, with
// device-coherent loads)
template <int BIAS2, int BN_, bool ADD = false>
__device__ __forceinline__ void store_tile(f32x16 (&acc)[TM][Tile<BN_>::TN], const int* sAlpha, const int* sBeta,
                                           float* C, int64_t ldc, int64_t M, int64_t N, int64_t m0, int64_t n0,
                                           int wm, int wn, int lane, bool split,
                                           const char* other_slot = nullptr, int wbase = 0) {
    constexpr int BN = BN_, WN = Tile<BN_>::WN, TN = Tile<BN_>::TN;
    const int64_t rowsC = min((int64_t)BM, M - m0), colsC = min((int64_t)BN, N - n0);
    const __amdgpu_buffer_rsrc_t rq =
        __builtin_amdgcn_make_buffer_rsrc((void*)other_slot, (short)0, ADD ? (int)BM * BN * 4 : 0, 0x00020000);
    if ((int64_t)BM * ldc <= ((int64_t)1 << 28)) {
        // buffer descriptor over the tile's rows of C: stores to rows past M fall outside it and
        // are dropped; columns past N are masked per lane (edge tiles only)
        const __amdgpu_buffer_rsrc_t rc = __builtin_amdgcn_make_buffer_rsrc(
            (void*)(C + m0 * ldc + n0), (short)0, (int)(((rowsC - 1) * ldc + colsC) * 4), 0x00020000);
        const int lrow = wm * WM + 4 * (lane >> 5);
        const int lcol = wn * WN + (lane & 31);
        const int voff = (lrow * (int)ldc + lcol) * 4;
        int beta[TN], bmax[TN];
        bool colok[TN];
#pragma unroll
        for (int tj = 0; tj < TN; tj++) {
            bmax[tj] = sBeta[lcol + 32 * tj];
            beta[tj] = bmax[tj] - BIAS2;
            colok[tj] = lcol + 32 * tj < colsC;
        }
        // one straight-line store sequence per case (split or not, edge columns or not)
        auto store_all = [&](auto split_c, auto edge_c) {
            constexpr bool SPLIT = decltype(split_c)::value, EDGE = decltype(edge_c)::value;
#pragma unroll
            for (int ti = 0; ti < TM; ti++)
#pragma unroll
                for (int g = 0; g < 4; g++) {
                    // row exponents of v = 4 g .. 4 g + 3 (four consecutive rows)
                    const int4 al = *reinterpret_cast<const int4*>(sAlpha + lrow + 32 * ti + 8 * g);
                    const int alr[4] = {al.x, al.y, al.z, al.w};
                    f32x4 other[TN];
                    if (ADD) {
#pragma unroll
                        for (int tj = 0; tj < TN; tj++)
                            other[tj] = __builtin_bit_cast(
                                f32x4, __builtin_amdgcn_raw_buffer_load_b128(rq, wbase + ((ti * 4 + tj) * 4 + g) * 1024,
                                                                             0, AUX_DEVICE_COHERENT));
                    }
#pragma unroll
                    for (int r = 0; r < 4; r++) {
                        const int soff = (32 * ti + 8 * g + r) * (int)ldc * 4;
#pragma unroll
                        for (int tj = 0; tj < TN; tj++) {
                            if (EDGE && !colok[tj]) continue;
                            float val = __builtin_amdgcn_ldexpf(acc[ti][tj][4 * g + r], alr[r] + beta[tj]);
                            if (ADD) val += other[tj][r];
                            val = poisoned(val, alr[r], bmax[tj]);
                            if (SPLIT)
                                __builtin_amdgcn_raw_ptr_buffer_atomic_fadd_f32(val, rc, voff + 128 * tj, soff, 0);
                            else
                                __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, val), rc,
                                                                      voff + 128 * tj, soff, 0);
                        }
                    }
                }
        };
        using T = std::true_type;
        using Fa = std::false_type;
        const bool edge = colsC < BN;
        if (split) {
            if (edge) store_all(T(), T());
            else store_all(T(), Fa());
        } else {
            if (edge) store_all(Fa(), T());
            else store_all(Fa(), Fa());
        }
    } else {
        // very wide C (ldc beyond 2^20): 64-bit addressing
#pragma unroll
        for (int ti = 0; ti < TM; ti++)
#pragma unroll
            for (int tj = 0; tj < TN; tj++) {
                const int lj = wn * WN + tj * 32 + (lane & 31);
                const int64_t gj = n0 + lj;
                const int beta = sBeta[lj];
#pragma unroll
                for (int v = 0; v < 16; v++) {
                    const int li = wm * WM + ti * 32 + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
                    const int64_t gi = m0 + li;
                    if (gi < M && gj < N) {
                        float val = __builtin_amdgcn_ldexpf(acc[ti][tj][v], sAlpha[li] + beta - BIAS2);
                        if (ADD)
                            val += __builtin_bit_cast(
                                float, __builtin_amdgcn_raw_buffer_load_b32(
                                           rq, wbase + ((ti * 4 + tj) * 4 + v / 4) * 1024 + 4 * (v % 4), 0,
                                           AUX_DEVICE_COHERENT));
                        val = poisoned(val, sAlpha[li], beta);
                        if (split) unsafeAtomicAdd(C + gi * ldc + gj, val);
                        else C[gi * ldc + gj] = val;
                    }
                }
            }
    }
}

template <class F, int BN_>
__global__ __launch_bounds__(NTHREADS) void gemm_kernel(
    const uint8_t* __restrict__ A, const int8_t* __restrict__ As,
    const uint8_t* __restrict__ B, const int8_t* __restrict__ Bs,
    int64_t M, int64_t N, int64_t K, float* __restrict__ C, int64_t ldc, int fidx, int64_t nsb, Div32 dgq) {
    using TL = Tile<BN_>;
    constexpr int BN = TL::BN, WN = TL::WN, TN = TL::TN, STAGE = TL::STAGE, TASKS = TL::TASKS;
    constexpr int PLANE_B = TL::PLANE_B;
    constexpr int MFMA_PER_SUB = TL::MFMA_PER_SUB, MPG = TL::MFMA_PER_GROUP;
    // static LDS (146 KB for 256 x 256 tiles): gfx950 has 160 KB per workgroup, and a static
    // array needs no per-device launch attribute
    __shared__ __attribute__((aligned(16))) char smem[TL::SMEM];
    const char* lut = smem;
    char* stage0 = smem + LUT_BYTES;
    char* stage1 = stage0 + STAGE;
    int* sAlpha = reinterpret_cast<int*>(smem + LUT_BYTES + 2 * STAGE);
    int* sBeta = sAlpha + BM;

    const int tid = threadIdx.x;
    {
        uint32_t* l = reinterpret_cast<uint32_t*>(smem);
        for (int i = tid; i < GEMM_DEC_ENTRIES * LUT_COPIES; i += NTHREADS) l[i] = g_dec[fidx][i / LUT_COPIES];
    }

    const int64_t m0 = (int64_t)blockIdx.y * BM, n0 = (int64_t)blockIdx.x * BN;
    const int64_t nkb = K / 32;
    // this workgroup's share of the K blocks (split-K over grid.z)
    const int64_t per = (nkb + gridDim.z - 1) / gridDim.z;
    const int64_t kb0 = (int64_t)blockIdx.z * per;
    const int64_t kb1 = min(nkb, kb0 + per);
    const int64_t nsteps = kb1 - kb0;
    const int64_t row_bytes = F::PACKED7 ? nkb * 28 : K;

    // buffer descriptors over the tile's rows (reads past the last row return zero)
    const int64_t rowsA = min((int64_t)BM, M - m0), rowsB = min((int64_t)BN, N - n0);
    const __amdgpu_buffer_rsrc_t rcA = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(A + m0 * row_bytes), (short)0, (int)(rowsA * row_bytes), 0x00020000);
    const __amdgpu_buffer_rsrc_t rcB = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(B + n0 * row_bytes), (short)0, (int)(rowsB * row_bytes), 0x00020000);
    // scales are read as aligned dwords (a 32-bit result keeps the compiler from extending a
    // byte at its load): the descriptors start at the dword below the tile's first scale and
    // end at the dword that holds its last one, all inside mapped pages
    // (nsb scales per row, one per G = 32 (G / 32) elements: K block kb has scale kb / (G / 32))
    const uintptr_t sa0 = reinterpret_cast<uintptr_t>(As + m0 * nsb), sb0 = reinterpret_cast<uintptr_t>(Bs + n0 * nsb);
    const int dA = (int)(sa0 & 3), dB = (int)(sb0 & 3);
    const __amdgpu_buffer_rsrc_t rsA = __builtin_amdgcn_make_buffer_rsrc(
        reinterpret_cast<void*>(sa0 - dA), (short)0, (int)((dA + rowsA * nsb + 3) & ~3), 0x00020000);
    const __amdgpu_buffer_rsrc_t rsB = __builtin_amdgcn_make_buffer_rsrc(
        reinterpret_cast<void*>(sb0 - dB), (short)0, (int)((dB + rowsB * nsb + 3) & ~3), 0x00020000);
    auto sidx = [&](int64_t kb) { return (int)div32((uint32_t)kb, dgq); };

    // expansion tasks: rows (tid >> 2) + 64 j of A (j < 4) and rows (tid >> 2) + 64 (j - 4) of B
    // (4 <= j < TASKS), chunk q = tid & 3
    const int q = tid & 3;
    const int r0 = tid >> 2;
    const int copy4 = (tid & (LUT_COPIES - 1)) * 4;
    const int off0 = swz(r0, q);                 // swz(r0 + 64 j, q) = off0 + 64 j * ROW_BYTES
    const int voff_code = (int)(r0 * row_bytes) + (F::PACKED7 ? 4 * ((7 * q) >> 2) : 8 * q);
    // byte offset of task j's scale of block kb: xA/xB + 64 (j & 3) nsb + sidx(kb), where the
    // middle term is a multiple of 4 and so moves only the dword
    const int xA = dA + (int)(r0 * nsb), xB = dB + (int)(r0 * nsb);
    // the row maxima of this thread's tasks, one byte each (scales lie in [-128, 127])
    uint32_t alpha_pk[2] = {0u, 0u};   // filled once the maxima are known
    auto alpha_of = [&](int j) { return (int)__builtin_amdgcn_sbfe(alpha_pk[j >> 2], 8 * (j & 3), 8); };
    auto task_dst_hi = [&](char* stage, int j) {
        return stage + (j < 4 ? 0 : 2 * PLANE) + off0 + 64 * (j & 3) * ROW_BYTES;
    };
    auto task_lo_plane = [](int j) { return j < 4 ? PLANE : PLANE_B; };   // hi -> lo plane distance

    // one register set of codes in flight: task j's codes of block kb+1 are loaded right after
    // its codes of block kb have been read, so each load has a whole step to arrive.  Loads are
    // unconditional (a block past the workgroup's range reads the next row, or zero past the
    // tile, and is never expanded).
    Raw<F> raw[TASKS];
    // per step: the block whose codes are read (cur) and the one requested (next)
    struct Blocks {
        int64_t next;
        int vA, vB;       // scale dword offsets of the next block, rows r0 of A and B
        int shA, shB;     // bit position of the scale byte in its dword, current block
    };
    auto blocks = [&](int64_t kb_cur) {
        Blocks b;
        b.next = kb_cur + 1;
        b.vA = (xA + sidx(b.next)) & ~3;
        b.vB = (xB + sidx(b.next)) & ~3;
        b.shA = 8 * ((xA + sidx(kb_cur)) & 3);
        b.shB = 8 * ((xB + sidx(kb_cur)) & 3);
        return b;
    };
    auto fetch = [&](int j, int64_t kb, int vscl) {
        const int ro = 64 * (j & 3);
        load_raw<F>(j < 4 ? rcA : rcB, j < 4 ? rsA : rsB, voff_code,
                    (int)(ro * row_bytes + kb * (F::PACKED7 ? 28 : 32)), vscl, (int)(ro * nsb), q, raw[j]);
    };
    // gather: task j's table entries into e, then the load of its next block; returns
    // D = (row maximum) - (block scale), and files min(D, 48) for the fixup pass
    uint32_t dpk[2];
    auto gather_task = [&](int j, const Blocks& b, uint32_t* e) {
        const Chunk c = settle<F>(raw[j], q, j < 4 ? b.shA : b.shB);
        fetch(j, b.next, j < 4 ? b.vA : b.vB);
        gather_chunk<F>(c, lut, copy4, e);
        const int D = alpha_of(j) - c.a;
        const uint32_t db = (uint32_t)min(D, 48) << (8 * (j & 3));
        dpk[j >> 2] = (j & 3) ? (dpk[j >> 2] | db) : db;
        return D;
    };
    // pack and scale; `need` collects blocks that the 24-binade multiplier cannot reach
    auto finish_task = [&](int D, char* stage, int j, const uint32_t* e, bool& need) {
        char* hd = task_dst_hi(stage, j);
        need |= D > 24;
        finish_chunk(e, D, hd, hd + task_lo_plane(j));
    };
    // rare second scaling pass (block more than 24 binades below its row's top)
    auto fixup = [&](char* stage, bool need) {
        if (__any(need)) {   // wave-uniform: taken only when some lane has such a block
#pragma unroll
            for (int j = 0; j < TASKS; j++) {
                const int D = (int)((dpk[j >> 2] >> (8 * (j & 3))) & 0xFFu);
                if (D > 24) {
                    char* hd = task_dst_hi(stage, j);
                    rescale_chunk(hd, D);
                    rescale_chunk(hd + task_lo_plane(j), D);
                }
            }
        }
    };

    // codes of block 0 are requested before the maxima are computed, so both latencies overlap
#pragma unroll
    for (int j = 0; j < TASKS; j++) fetch(j, kb0, j < 4 ? (xA + sidx(kb0)) & ~3 : (xB + sidx(kb0)) & ~3);

    // largest block scale of every A and B row of the tile (over all of K), 0 for rows past the
    // edge: one row per thread; up to 15 unaligned bytes at each end, 16-byte loads in between,
    // eight of them in flight per round
    auto row_max = [](const int8_t* sp, int n) {
        int m = -128;
        auto max4 = [&](uint32_t w) {
#pragma unroll
            for (int bb = 0; bb < 4; bb++) m = max(m, scale_key((int)(int8_t)(w >> (8 * bb))));
        };
        const int head = min((int)((16 - (reinterpret_cast<uintptr_t>(sp) & 15)) & 15), n);
        const int nch = (n - head) >> 4;
        const int tail = n - head - 16 * nch;
        int hb[15], tb[15];
#pragma unroll
        for (int i = 0; i < 15; i++) {
            hb[i] = i < head ? scale_key((int)sp[i]) : -127;
            tb[i] = i < tail ? scale_key((int)sp[head + 16 * nch + i]) : -127;
        }
        const uint4* ab = reinterpret_cast<const uint4*>(sp + head);
        for (int c = 0; c < nch; c += 8) {
            uint4 v[8];
#pragma unroll
            // padding of -127: below or at every real key (scales are at least -127, -128 is the key)
            for (int u = 0; u < 8; u++) v[u] = c + u < nch ? ab[c + u] : make_uint4(0x81818181u, 0x81818181u, 0x81818181u, 0x81818181u);
#pragma unroll
            for (int u = 0; u < 8; u++) {
                max4(v[u].x);
                max4(v[u].y);
                max4(v[u].z);
                max4(v[u].w);
            }
        }
#pragma unroll
        for (int i = 0; i < 15; i++) m = max(m, max(hb[i], tb[i]));
        return m;
    };
    sAlpha[tid] = tid < rowsA ? row_max(As + (m0 + tid) * nsb, (int)nsb) : 0;
    if (tid < BN) sBeta[tid] = tid < rowsB ? row_max(Bs + (n0 + tid) * nsb, (int)nsb) : 0;
    __syncthreads();

#pragma unroll
    for (int j = 0; j < TASKS; j++) {
        // a poisoned row expands against the largest scale (every offset D = 127 - a stays in
        // [0, 255]); its outputs are NaN whatever it accumulates
        const int am = j < 4 ? sAlpha[r0 + 64 * j] : sBeta[r0 + 64 * (j - 4)];
        const int al = am >= POISON_KEY ? 127 : am;
        alpha_pk[j >> 2] |= ((uint32_t)al & 0xFFu) << (8 * (j & 3));
    }

    const int lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    // lane part of a fragment address: row (lane & 31) of a 32-row tile, chunk 2 kq + (lane >> 5);
    // the swizzle only depends on bits 1..3 of the row, which the tile bases leave alone
    const int lr = lane & 31;
    const int fsw = ((lr >> 1) ^ (lr >> 3)) & 3;
    const int foff0 = lr * ROW_BYTES + 16 * ((0 + (lane >> 5)) ^ fsw);
    const int foff1 = lr * ROW_BYTES + 16 * ((2 + (lane >> 5)) ^ fsw);
    const int abase = wm * WM * ROW_BYTES, bbase = 2 * PLANE + wn * WN * ROW_BYTES;
    auto load_frag = [&](Frag<TN>& f, const char* st, int kq) {
        const char* pa = st + abase + (kq ? foff1 : foff0);
        const char* pb = st + bbase + (kq ? foff1 : foff0);
#pragma unroll
        for (int t = 0; t < TM; t++) {
            f.ah[t] = *reinterpret_cast<const half8*>(pa + t * 32 * ROW_BYTES);
            f.al[t] = *reinterpret_cast<const half8*>(pa + PLANE + t * 32 * ROW_BYTES);
        }
#pragma unroll
        for (int t = 0; t < TN; t++) {
            f.bh[t] = *reinterpret_cast<const half8*>(pb + t * 32 * ROW_BYTES);
            f.bl[t] = *reinterpret_cast<const half8*>(pb + PLANE_B + t * 32 * ROW_BYTES);
        }
    };

    f32x16 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; i++)
#pragma unroll
        for (int j = 0; j < TN; j++)
#pragma unroll
            for (int v = 0; v < 16; v++) acc[i][j][v] = 0.f;

    // MFMA number idx (0..47) of a half step: product p = idx / 16 over the 4 x 4 tiles
    // MFMA number idx (0 .. MFMA_PER_SUB-1) of a slice: product p = idx / (TM TN) over the tiles
    // within a product (hi.hi, hi.lo, lo.hi) the 16 tiles go in snake order over (i, j), so
    // consecutive MFMAs share an operand fragment (less switching in the matrix cores: 0.7% faster
    // at the power limit); each accumulator still takes the three products 16 MFMAs apart, in the
    // same order, so C does not change
    auto mfma = [&](const Frag<TN>& f, int idx) {
        const int p = idx / (TM * TN), i = (idx / TN) % TM, j = (i & 1) ? TN - 1 - idx % TN : idx % TN;
        const half8& a = (p == 2) ? f.al[i] : f.ah[i];
        const half8& b = (p == 1) ? f.bl[j] : f.bh[j];
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, acc[i][j], 0, 0, 0);
    };

    // prologue: expand block 0 (requesting block 1), fragments of its first half
    Frag<TN> f0, f1;
    {
        const Blocks b0 = blocks(kb0);
        bool need = false;
#pragma unroll
        for (int j = 0; j < TASKS; j++) {
            uint32_t e[8];
            const int D = gather_task(j, b0, e);
            finish_task(D, stage0, j, e, need);
        }
        fixup(stage0, need);
    }
    __syncthreads();
    load_frag(f0, stage0, 0);

    // one step with a successor: MFMAs of step s from `cur` (f0 already loaded); step s+1 is
    // expanded into `nxt` while the MFMAs run, and the codes of step s+2 are requested
    auto step = [&](int64_t s, const char* cur, char* nxt) {
        const Blocks b = blocks(kb0 + s + 1);
        load_frag(f1, cur, 1);
        uint32_t e0[8], e1[8];
        int D0 = 0, D1 = 0;
        bool need = false;
        D0 = gather_task(0, b, e0);
        // TASKS groups of MPG MFMAs (slice 0 from f0, then slice 1 from f1); group g gathers
        // task g+1 and packs task g; the barrier sits before the last group so the next step's
        // fragments load behind its MFMAs
#pragma unroll
        for (int g = 0; g < TASKS - 1; g++) {
#pragma unroll
            for (int m = 0; m < MPG; m++) {
                const int gi = g * MPG + m;
                mfma(gi < MFMA_PER_SUB ? f0 : f1, gi % MFMA_PER_SUB);
            }
            ((g & 1) ? D0 : D1) = gather_task(g + 1, b, (g & 1) ? e0 : e1);
            finish_task((g & 1) ? D1 : D0, nxt, g, (g & 1) ? e1 : e0, need);
#pragma unroll
            for (int m = 0; m < MPG; m++) {
                __builtin_amdgcn_sched_group_barrier(SG_MFMA, 1, 0);
                __builtin_amdgcn_sched_group_barrier(SG_VALU, 3, 0);
                __builtin_amdgcn_sched_group_barrier(SG_DS_RD, 1, 0);
            }
            __builtin_amdgcn_sched_barrier(0);
        }
        finish_task((TASKS & 1) ? D0 : D1, nxt, TASKS - 1, (TASKS & 1) ? e0 : e1, need);
        fixup(nxt, need);
        __syncthreads();
        load_frag(f0, nxt, 0);
#pragma unroll
        for (int m = MFMA_PER_SUB - MPG; m < MFMA_PER_SUB; m++) mfma(f1, m);
    };

    char* cur = stage0;
    char* nxt = stage1;
    for (int64_t s = 0; s + 1 < nsteps; s++) {
        step(s, cur, nxt);
        char* t = cur;
        cur = nxt;
        nxt = t;
    }
    // the last step: MFMAs only
    load_frag(f1, cur, 1);
#pragma unroll
    for (int m = 0; m < MFMA_PER_SUB; m++) mfma(f0, m);
#pragma unroll
    for (int m = 0; m < MFMA_PER_SUB; m++) mfma(f1, m);

    store_tile<2 * F::GEMM_BIAS, BN>(acc, sAlpha, sBeta, C, ldc, M, N, m0, n0, wm, wn, lane, gridDim.z > 1);
}

// zero-fill of the output rows (split-K accumulates into C)
__global__ __launch_bounds__(256) void zero_rows_kernel(float* __restrict__ C, int64_t M, int64_t N, int64_t ldc) {
    const int64_t total = M * N;
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < total; i += (int64_t)gridDim.x * 256) {
        const int64_t r = i / N;
        C[r * ldc + (i - r * N)] = 0.f;
    }
}

// ---------------------------------------------------------------------------------------------
// Workspace path.  The codes of A and B are expanded once, by their own kernels, into fp16
// (hi, lo) planes laid out exactly like the LDS stages above; the GEMM then streams each
// 64 KB stage into LDS with buffer-to-LDS loads and its main loop is left to the MFMAs.
// The expanded values are those of the fused kernel, and the MFMA order is the same, so both
// paths give the same C bit for bit.

// workspace of one GEMM: per operand with R rows, RT = ceil(R / 256) row tiles, nkb = K / 32
//   planes [nkb][RT][hi, lo][256 rows][64 B] (32 KB per (kb, rt), rows swizzled as in a stage,
//          zero past R)
//   maxima [RT * 256] int32 (largest block scale of each row, 0 past R)
// K is split in two when the tiles cover fewer than the 256 compute units and K is long enough:
// each half writes its scaled 256 x 256 partial tile to the workspace, and the half that
// finishes last adds the other's to its own and stores C (a per-tile arrival counter decides)
constexpr int64_t PART_BYTES = (int64_t)BM * 256 * 4;

struct WsLayout {
    int64_t rta, rtb, planes_a, planes_b, max_a, max_b, cnt, part, bytes;
    int splits;
};

WsLayout ws_layout(int64_t M, int64_t N, int64_t K) {
    WsLayout w;
    const int64_t nkb = K / 32;
    w.rta = (M + BM - 1) / BM;
    w.rtb = (N + BM - 1) / BM;
    const int64_t tiles = w.rta * w.rtb;
    w.splits = (tiles < 256 && nkb >= 16) ? 2 : 1;
    w.planes_a = 0;
    w.planes_b = w.planes_a + nkb * w.rta * 2 * PLANE;
    w.max_a = w.planes_b + nkb * w.rtb * 2 * PLANE;
    w.max_b = w.max_a + w.rta * BM * 4;
    int64_t end = w.max_b + w.rtb * BM * 4;
    w.cnt = w.part = end;
    if (w.splits > 1) {
        w.cnt = (end + 255) & ~(int64_t)255;
        w.part = w.cnt + ((tiles * 4 + 255) & ~(int64_t)255);
        end = w.part + tiles * w.splits * PART_BYTES;
    }
    w.bytes = end;
    return w;
}

// one launch before the expansion: row maxima of the block scales of A (workgroups
// [0, ga)) and of B ([ga, ga + gb)), 16 lanes per row, each over every 16th of the row's nsb
// scales; one more workgroup zeroes the per-tile arrival counters when K is split
__global__ __launch_bounds__(256) void prep_kernel(const int8_t* __restrict__ as, const int8_t* __restrict__ bs,
                                                   int64_t M, int64_t N, int64_t nsb, int ga, int gb,
                                                   int* __restrict__ maxA, int* __restrict__ maxB,
                                                   int* __restrict__ cnt, int ncnt) {
    const int bid = (int)blockIdx.x;
    if (bid >= ga + gb) {
        for (int i = threadIdx.x; i < ncnt; i += 256) cnt[i] = 0;
        return;
    }
    const bool isA = bid < ga;
    const int8_t* s = isA ? as : bs;
    const int64_t R = isA ? M : N;
    int* out = isA ? maxA : maxB;
    const int64_t row = (int64_t)(isA ? bid : bid - ga) * 16 + (threadIdx.x >> 4);
    const int part = threadIdx.x & 15;
    int m = -128;
    if (row < R) {
        const int8_t* sp = s + row * nsb;
#pragma unroll 8
        for (int64_t sb = part; sb < nsb; sb += 16) m = max(m, scale_key((int)sp[sb]));
    }
#pragma unroll
    for (int o = 8; o > 0; o >>= 1) m = max(m, __shfl_xor(m, o, 16));
    if (part == 0) out[row] = row < R ? m : 0;   // the grid covers exactly the padded rows
}

// expansion of 64 rows x 4 K-blocks per workgroup: thread = (row (t >> 2) of the group, chunk
// q = t & 3), one task per block; the same table values and multipliers as the fused kernel
struct ExpandOperand {
    const uint8_t* codes;
    const int8_t* scales;
    int64_t rows, tiles;      // rows, and row tiles of 256
    const int* rmax;          // row maxima (keys of the block scales), from prep_kernel
    char* planes;
    int fidx;                 // format: which expansion table
    int64_t nsb;              // scales per row (K / G)
    Div32 dgq;                // K block kb has scale kb / (G / 32)
};

// both operands in one launch: workgroups [0, 4 A.tiles) take A, the rest B (F fixes the code
// packing, which both share; each operand brings its own table)
// The row maxima come from prep_kernel (one launch over the scales): taking them inside the
// expansion instead, by every K group over the whole row, measured slower on the large shapes
// (8192 x 14336 x 4096: 118 us against 87 + 4 us) and even on 2048 x 4096 x 4096.
template <class F>
__global__ __launch_bounds__(256) void expand_kernel(ExpandOperand opA, ExpandOperand opB, int64_t nkb) {
    __shared__ uint32_t lut[GEMM_DEC_ENTRIES];
    const bool isA = (int64_t)blockIdx.x < 4 * opA.tiles;
    const ExpandOperand& op = isA ? opA : opB;
    lut[threadIdx.x] = g_dec[op.fidx][threadIdx.x];
    const uint8_t* X = op.codes;
    const int8_t* Xs = op.scales;
    const int64_t R = op.rows, RT = op.tiles;
    char* planes = op.planes;
    const int64_t row_bytes = F::PACKED7 ? nkb * 28 : nkb * 32;
    const int64_t r0 = (int64_t)(isA ? blockIdx.x : blockIdx.x - 4 * opA.tiles) * 64;
    const int64_t kbase = (int64_t)blockIdx.y * 4;
    const int lr = threadIdx.x >> 2, q = threadIdx.x & 3;
    const int64_t row = r0 + lr;
    // buffer descriptors over the group's rows (none past R: those tasks read zeros)
    const int64_t rg = max((int64_t)0, min((int64_t)64, R - r0));
    const __amdgpu_buffer_rsrc_t rc = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(X + min(r0, R) * row_bytes), (short)0, (int)(rg * row_bytes), 0x00020000);
    const int64_t nsb = op.nsb;
    const uintptr_t s0 = reinterpret_cast<uintptr_t>(Xs + min(r0, R) * nsb);
    const int ds = (int)(s0 & 3);
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
        reinterpret_cast<void*>(s0 - ds), (short)0, (int)((ds + rg * nsb + 3) & ~3), 0x00020000);
    const int voff_code = (int)(lr * row_bytes) + (F::PACKED7 ? 4 * ((7 * q) >> 2) : 8 * q);
    const int x = ds + (int)(lr * nsb);   // byte offset of the row's scales in rs
    auto sidx = [&](int64_t kb) { return (int)div32((uint32_t)kb, op.dgq); };
    Raw<F> raw[4];
#pragma unroll
    for (int t = 0; t < 4; t++)
        load_raw<F>(rc, rs, voff_code, (int)((kbase + t) * (F::PACKED7 ? 28 : 32)), (x + sidx(kbase + t)) & ~3, 0, q,
                    raw[t]);
    const int alpha = op.rmax[row];   // the padded rows hold 0
    __syncthreads();
#pragma unroll
    for (int t = 0; t < 4; t++) {
        const int64_t kb = kbase + t;
        if (kb >= nkb) break;
        const Chunk c = settle<F>(raw[t], q, 8 * ((x + sidx(kb)) & 3));
        uint32_t e[8];
#pragma unroll
        for (int i = 0; i < 8; i++) e[i] = lut[chunk_code<F>(c, i)];
        uint32_t hv[4], lv[4];
        expand_chunk8(e, alpha - c.a, hv, lv);
        char* dst = planes + (kb * RT + row / BM) * (2 * PLANE) + swz((int)(row % BM), q);
        *reinterpret_cast<uint4*>(dst) = make_uint4(hv[0], hv[1], hv[2], hv[3]);
        *reinterpret_cast<uint4*>(dst + PLANE) = make_uint4(lv[0], lv[1], lv[2], lv[3]);
    }
}

// Work item of a workgroup on 8 XCDs.  Workgroups go to the XCDs round robin (linear id mod 8),
// and each XCD has its own L2: XCD x takes the x-th eighth of the work items, in an order that
// walks groups of 4 tile rows column by column, so the workgroups resident on one XCD at a time
// cover a compact block of tiles and share their A and B stages in its L2.
struct WorkItem {
    int ty, tx, split;
    bool valid;
};

__device__ __forceinline__ WorkItem work_item(int tiles_y, int tiles_x, int splits) {
    constexpr int XCDS = 8, GROUP = 4;
    const int total = tiles_y * tiles_x * splits;
    const int share = (total + XCDS - 1) / XCDS;
    const int lin = (int)blockIdx.x;
    const int u = (lin % XCDS) * share + lin / XCDS;
    WorkItem w;
    w.valid = u < total;
    const int t = u / splits;
    w.split = u - t * splits;
    const int g = t / (GROUP * tiles_x);
    const int gh = min(GROUP, tiles_y - g * GROUP);
    const int local = t - g * GROUP * tiles_x;
    w.ty = g * GROUP + local % gh;
    w.tx = local / gh;
    return w;
}

// ---------------------------------------------------------------------------------------------
// Output requantization (Sec. 3.2: products are closed on widened coordinates; only the explicit
// requantization to a finite destination may saturate).  The tile's fp32 values, exactly those
// store_tile would write, are quantized in blocks of G (32, 64, 128 or 256) along each output row
// by the quantizer's rule (codec.hpp), so the codes equal curvefp_quantize of curvefp_gemm_ws's C
// with that block, bit for bit.  The tile goes through LDS (the freed stages) in four slices of
// 64 rows: every wave writes its fp32 values of the slice (the 32 rows ti of both wave rows),
// then each thread quantizes two groups of 32 of the slice (a block's G/32 groups sit in
// adjacent lanes and share its maximum) and stores their codes (32 contiguous bytes, or 28
// packed) and the block's scale.
// The accumulators are only ever indexed by unrolled loop counters.
struct ReqOut {
    uint8_t* codes;        // [M][N] bytes, or [M][N/32][28] for 7-bit codes
    int8_t* scales;        // [M][N/G]
    QRule rule;
    int fmt;               // output format (table row)
    int packed7;
    int glog;              // output blocks of G = 32 << glog elements along each row (G <= 256)
};

// float offset of (row, col) in a 64 x 256 fp32 slice: 16-byte chunks XOR-swizzled by row & 7,
// so a thread reading its block's eight chunks and the lanes of a wave spread over the banks
__device__ __forceinline__ int slice_off(int row, int col) {
    return row * 256 + ((((col >> 2) ^ (row & 7))) << 2) + (col & 3);
}

template <int BIAS2, bool ADD>
__device__ __forceinline__ void requant_tile(f32x16 (&acc)[TM][4], const int* sAlpha, const int* sBeta,
                                             int64_t M, int64_t N, int64_t m0, int64_t n0, int wm, int wn,
                                             int lane, int tid, const char* other_slot, int wbase, char* slice_mem,
                                             char* aux, const ReqOut& ro) {
    constexpr int BN = 256, WN = Tile<256>::WN, TN = Tile<256>::TN;
    float* slice = reinterpret_cast<float*>(slice_mem);          // 64 rows x 256 fp32 (64 KB)
    // the output format's table behind one octave of rank-0 entries (base 0, threshold 0xFFFF):
    // a magnitude scaled by ldexp lands in the pad or below it exactly when the quantizer's
    // rule gives it rank 0, so the lookup needs no range tests
    uint32_t* qlut = reinterpret_cast<uint32_t*>(aux);
    const QRule q = ro.rule;
    __syncthreads();                                             // every wave is done with the stages
    for (int i = tid; i < q.qsize + 128; i += NTHREADS) qlut[i] = i < 128 ? 0xFFFFu : g_gq_lut[ro.fmt][i - 128];
    const int ibase = (126 + q.oz) << 7, itop = q.qsize + 127;
    const __amdgpu_buffer_rsrc_t rq =
        __builtin_amdgcn_make_buffer_rsrc((void*)other_slot, (short)0, ADD ? (int)BM * BN * 4 : 0, 0x00020000);
    const int lrow = 4 * (lane >> 5);                            // row of the lane within a 32-row block
    const int lcol = wn * WN + (lane & 31);
    const int64_t nbr = N / 32;                                  // output blocks per row
#pragma unroll
    for (int ti = 0; ti < TM; ti++) {
        // phase A: this wave's 32 rows of slice ti (slice rows wm * 32 ..) into LDS; the other
        // K half's sixteen partial vectors are all requested before the first is used
        f32x4 other[TN][4];
        if (ADD) {
#pragma unroll
            for (int tj = 0; tj < TN; tj++)
#pragma unroll
                for (int g = 0; g < 4; g++)
                    other[tj][g] = __builtin_bit_cast(
                        f32x4, __builtin_amdgcn_raw_buffer_load_b128(rq, wbase + ((ti * 4 + tj) * 4 + g) * 1024, 0,
                                                                     AUX_DEVICE_COHERENT));
        }
#pragma unroll
        for (int tj = 0; tj < TN; tj++) {
            const int beta = sBeta[lcol + 32 * tj] - BIAS2;
#pragma unroll
            for (int g = 0; g < 4; g++) {
                const int4 al = *reinterpret_cast<const int4*>(sAlpha + wm * WM + 32 * ti + lrow + 8 * g);
                const int alr[4] = {al.x, al.y, al.z, al.w};
#pragma unroll
                for (int r = 0; r < 4; r++) {
                    float val = __builtin_amdgcn_ldexpf(acc[ti][tj][4 * g + r], alr[r] + beta);
                    if (ADD) val += other[tj][g][r];
                    val = poisoned(val, alr[r], beta + BIAS2);
                    slice[slice_off(wm * 32 + lrow + 8 * g + r, lcol + 32 * tj)] = val;
                }
            }
        }
        __syncthreads();
        // phase B: 64 rows x 8 groups of 32, two per thread (eight adjacent lanes cover one row,
        // so a block of G = 32 << glog is G/32 adjacent lanes)
        for (int bi = tid; bi < 64 * 8; bi += NTHREADS) {
            const int srow = bi >> 3, cb = bi & 7;
            const int64_t row = m0 + (srow >> 5) * WM + 32 * ti + (srow & 31);
            const int64_t blk = n0 / 32 + cb;
            // groups past M or N hold zeros; blocks never straddle N (N % G == 0), and every lane
            // takes part in the block maximum before the invalid ones stop
            const bool valid = row < M && blk < nbr;
            // pass 1: the block maximum; pass 2: each 16-byte chunk (re-read from LDS) quantized
            // and packed into the output words, so only one chunk is held at a time
            const float* rowp = slice + srow * 256;
            auto chunk = [&](int c) {
                return *reinterpret_cast<const uint4*>(rowp + (((8 * cb + c) ^ (srow & 7)) << 2));
            };
            uint32_t amax = 0;
#pragma unroll
            for (int c = 0; c < 8; c++) {
                const uint4 v = chunk(c);
                amax = max(max(amax, max(v.x & 0x7FFFFFFFu, v.y & 0x7FFFFFFFu)),
                           max(v.z & 0x7FFFFFFFu, v.w & 0x7FFFFFFFu));
            }
            for (int o = 1; o < (1 << ro.glog); o <<= 1) amax = max(amax, (uint32_t)__shfl_xor((int)amax, o));
            if (!valid) continue;
            const int a = qr_scale(amax, q);
            // the packing is chosen once per block, so each loop below is straight-line code and
            // its table lookups can be scheduled together
            auto codes_of = [&](auto p7c) {
                constexpr bool P7 = decltype(p7c)::value;
                uint32_t wd[8] = {0, 0, 0, 0, 0, 0, 0, 0};
#pragma unroll
                for (int c = 0; c < 8; c++) {
                    const uint4 v = chunk(c);
                    const uint32_t b4[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
                    for (int j = 0; j < 4; j++) {
                        // |x| 2^-a by v_ldexp_f32: exact wherever it can reach a nonzero level
                        // (fp32 denormals are kept), below that it only needs to stay small
                        const uint32_t yb = __builtin_bit_cast(
                            uint32_t, __builtin_amdgcn_ldexpf(__builtin_bit_cast(float, b4[j] & 0x7FFFFFFFu), -a));
                        const uint32_t e = qlut[min(max((int)(yb >> 16) - ibase, 0), itop)];
                        const uint32_t rk = (e >> 16) + (((yb & 0xFFFFu) > (e & 0xFFFFu)) ? 1u : 0u);
                        const uint32_t code = rk | ((rk != 0 ? b4[j] >> 31 : 0u) << q.ec);
                        if (!P7) {
                            wd[c] |= code << (8 * j);
                        } else {
                            const int bit = 7 * (4 * c + j);
                            wd[bit >> 5] |= code << (bit & 31);
                            if ((bit & 31) > 25) wd[(bit >> 5) + 1] |= code >> (32 - (bit & 31));
                        }
                    }
                }
                // a block that held a NaN or an infinity (scale -128) keeps zero codes
                const uint32_t keep = a == -128 ? 0u : ~0u;
#pragma unroll
                for (int t = 0; t < 8; t++) wd[t] &= keep;
                if (!P7) {
                    uint4* dst = reinterpret_cast<uint4*>(ro.codes + row * N + 32 * blk);
                    dst[0] = make_uint4(wd[0], wd[1], wd[2], wd[3]);
                    dst[1] = make_uint4(wd[4], wd[5], wd[6], wd[7]);
                } else {
                    uint32_t* dst = reinterpret_cast<uint32_t*>(ro.codes + (row * nbr + blk) * 28);
#pragma unroll
                    for (int j = 0; j < 7; j++) dst[j] = wd[j];
                }
            };
            if (ro.packed7) codes_of(std::true_type());
            else codes_of(std::false_type());
            if ((cb & ((1 << ro.glog) - 1)) == 0) ro.scales[row * (nbr >> ro.glog) + (blk >> ro.glog)] = (int8_t)a;
        }
        __syncthreads();                                         // the slice is free for the next ti
    }
}

// GEMM on expanded planes: 256 x 256 tile per 256-thread workgroup as in the fused kernel (the
// same MFMA order, so the same C bit for bit).  Two LDS stages; a step (one K block) is
//   phase 1: the block's second fragment slice is read from LDS under the first slice's MFMAs;
//   barrier: every wave is done with the stage of this block, and the copy of the next block
//            into the other stage has landed;
//   phase 2: the copy of block s+2 into the stage just freed (buffer-to-LDS loads, 16 per
//            thread) and the reads of block s+1's first slice go out under the second slice's MFMAs.
// So each copy has a whole step to land, and the scheduler is held to this interleaving.
template <int BIAS2, bool REQ = false>
__global__ __launch_bounds__(NTHREADS) void gemm_ws_kernel(
    const char* __restrict__ PA, const char* __restrict__ PB, const int* __restrict__ maxA,
    const int* __restrict__ maxB, int64_t M, int64_t N, int64_t K, int64_t RTA, int64_t RTB,
    float* __restrict__ C, int64_t ldc, int splits, char* __restrict__ part, int* __restrict__ cnt,
    ReqOut ro) {
    using TL = Tile<256>;
    constexpr int BN = TL::BN, WN = TL::WN, TN = TL::TN, STAGE = TL::STAGE;
    constexpr int MPS = TL::MFMA_PER_SUB;   // 48 MFMAs per 16-wide K slice
    static_assert(TM == 4 && TN == 4 && MPS == 48, "the interleaving below assumes 4 x 4 MFMA tiles");
    // two stages as separate arrays: the loop below is unrolled so that every access names its
    // stage statically, and the compiler can see that copies into one stage and fragment reads
    // from the other do not overlap (so it may interleave them freely)
    __shared__ __attribute__((aligned(16))) char st0[STAGE];
    __shared__ __attribute__((aligned(16))) char st1[STAGE];
    __shared__ __attribute__((aligned(16))) int sAB[BM + BN + 4];
    int* sAlpha = sAB;
    int* sBeta = sAB + BM;
    int* sLast = sAB + BM + BN;

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const WorkItem wi = work_item((int)RTA, (int)RTB, splits);
    if (!wi.valid) return;   // the last XCD's share can run past the end (uniform per workgroup)
    const int64_t m0 = (int64_t)wi.ty * BM, n0 = (int64_t)wi.tx * BN;
    const int64_t nkb = K / 32;
    const int64_t per = (nkb + splits - 1) / splits;
    const int64_t kb0 = (int64_t)wi.split * per;
    const int64_t kb1 = min(nkb, kb0 + per);
    const int64_t nsteps = kb1 - kb0;
    sAlpha[tid] = maxA[m0 + tid];
    sBeta[tid] = maxB[n0 + tid];

    // stage of block kb in st: A's 32 KB then B's 32 KB, each a contiguous workspace
    // block; wave w copies kilobytes 8 w .. 8 w + 7 of each (lane l moves bytes 16 l .. 16 l + 15
    // of a kilobyte; the LDS address is M0 + 16 l)
    using lds_ptr = __attribute__((address_space(3))) void*;
    const int voff = 16 * lane;
    auto dma = [&](int64_t kb, char* st) {
        const __amdgpu_buffer_rsrc_t ra = __builtin_amdgcn_make_buffer_rsrc(
            (void*)(PA + (kb * RTA + wi.ty) * (2 * PLANE)), (short)0, 2 * PLANE, 0x00020000);
        const __amdgpu_buffer_rsrc_t rb = __builtin_amdgcn_make_buffer_rsrc(
            (void*)(PB + (kb * RTB + wi.tx) * (2 * PLANE)), (short)0, 2 * PLANE, 0x00020000);
#pragma unroll
        for (int i = 0; i < 8; i++) {
            const int kbyte = (wave * 8 + i) * 1024;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, (lds_ptr)(st + kbyte), 16, voff, kbyte, 0, 0);
            __builtin_amdgcn_raw_ptr_buffer_load_lds(rb, (lds_ptr)(st + 2 * PLANE + kbyte), 16, voff, kbyte, 0, 0);
        }
    };
    // this wave's copies have landed (vmcnt 0; the other counters left alone)
    auto dma_wait = [] { __builtin_amdgcn_s_waitcnt(0x0F70); };

    const int wm = (tid >> 6) >> 1, wn = (tid >> 6) & 1;
    const int lr = lane & 31;
    const int fsw = ((lr >> 1) ^ (lr >> 3)) & 3;
    const int foff0 = lr * ROW_BYTES + 16 * ((0 + (lane >> 5)) ^ fsw);
    const int foff1 = lr * ROW_BYTES + 16 * ((2 + (lane >> 5)) ^ fsw);
    const int abase = wm * WM * ROW_BYTES, bbase = 2 * PLANE + wn * WN * ROW_BYTES;
    // fragment reads in the order the MFMAs consume them (hi x hi by rows of A, then B lo, then A lo)
    auto load_frag = [&](Frag<TN>& f, const char* st, int kq) {
        const char* pa = st + abase + (kq ? foff1 : foff0);
        const char* pb = st + bbase + (kq ? foff1 : foff0);
        f.ah[0] = *reinterpret_cast<const half8*>(pa);
#pragma unroll
        for (int t = 0; t < TN; t++) f.bh[t] = *reinterpret_cast<const half8*>(pb + t * 32 * ROW_BYTES);
#pragma unroll
        for (int t = 1; t < TM; t++) f.ah[t] = *reinterpret_cast<const half8*>(pa + t * 32 * ROW_BYTES);
#pragma unroll
        for (int t = 0; t < TN; t++)
            f.bl[t] = *reinterpret_cast<const half8*>(pb + TL::PLANE_B + t * 32 * ROW_BYTES);
#pragma unroll
        for (int t = 0; t < TM; t++) f.al[t] = *reinterpret_cast<const half8*>(pa + PLANE + t * 32 * ROW_BYTES);
    };
    f32x16 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; i++)
#pragma unroll
        for (int j = 0; j < TN; j++)
#pragma unroll
            for (int v = 0; v < 16; v++) acc[i][j][v] = 0.f;
    // within a product (hi.hi, hi.lo, lo.hi) the 16 tiles go in snake order over (i, j), so
    // consecutive MFMAs share an operand fragment (less switching in the matrix cores: 0.7% faster
    // at the power limit); each accumulator still takes the three products 16 MFMAs apart, in the
    // same order, so C does not change
    auto mfma = [&](const Frag<TN>& f, int idx) {
        const int p = idx / (TM * TN), i = (idx / TN) % TM, j = (i & 1) ? TN - 1 - idx % TN : idx % TN;
        const half8& a = (p == 2) ? f.al[i] : f.ah[i];
        const half8& b = (p == 1) ? f.bl[j] : f.bh[j];
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, acc[i][j], 0, 0, 0);
    };
    // scheduling masks: MFMA, VMEM, DS read
    constexpr int SG_MFMA = 0x008, SG_VMEM = 0x010, SG_DSR = 0x100;

    // phase 1 of the step on the stage at st: one fragment read per two MFMAs over the first 32
    auto phase1 = [&](Frag<TN>& fa, Frag<TN>& fb, char* st) {
        // fa's reads went out a phase ago: waiting for them here costs nothing, and tells the
        // compiler that none is outstanding (else it waits for the first read below as well)
        __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0)
        load_frag(fb, st, 1);
#pragma unroll
        for (int m = 0; m < MPS; m++) mfma(fa, m);
#pragma unroll
        for (int i = 0; i < 16; i++) {
            __builtin_amdgcn_sched_group_barrier(SG_DSR, 1, 0);
            __builtin_amdgcn_sched_group_barrier(SG_MFMA, 2, 0);
        }
        __builtin_amdgcn_sched_group_barrier(SG_MFMA, MPS - 32, 0);
        __builtin_amdgcn_sched_barrier(0);
    };
    // the barrier between the phases
    auto handover = [&] {
        dma_wait();
        __syncthreads();
        __builtin_amdgcn_sched_barrier(0);
    };
    // phase 2: (with copy) block kb copied into the stage st and the next block's first slice
    // read from nx, one read and one copy per three MFMAs over all 48 (the copies' LDS writes
    // spread out, so they hold up the fragment reads less: 0.8% faster than one of each per two
    // MFMAs over the first 32, the same C)
    auto phase2 = [&](Frag<TN>& fa, Frag<TN>& fb, char* nx, bool copy, int64_t kb, char* st) {
        if (copy) dma(kb, st);
        load_frag(fa, nx, 0);
#pragma unroll
        for (int m = 0; m < MPS; m++) mfma(fb, m);
#pragma unroll
        for (int i = 0; i < 16; i++) {
            __builtin_amdgcn_sched_group_barrier(SG_DSR, 1, 0);
            if (copy) __builtin_amdgcn_sched_group_barrier(SG_VMEM, 1, 0);
            __builtin_amdgcn_sched_group_barrier(SG_MFMA, 3, 0);
        }
        __builtin_amdgcn_sched_barrier(0);
    };
    // a step that copies block kb into its own stage once done with it; one that copies
    // nothing; the last step (no barrier)
    Frag<TN> f0, f1;
    auto step_copy = [&](char* cur, char* nxt, int64_t kb) {
        phase1(f0, f1, cur);
        handover();
        phase2(f0, f1, nxt, true, kb, cur);
    };
    auto step_nocopy = [&](char* cur, char* nxt) {
        phase1(f0, f1, cur);
        handover();
        phase2(f0, f1, nxt, false, 0, cur);
    };
    auto step_final = [&](char* cur) {
        phase1(f0, f1, cur);
#pragma unroll
        for (int m = 0; m < MPS; m++) mfma(f1, m);
    };

    // stages alternate, and the last two steps always run on st0 then st1: with an odd step
    // count the first block goes to st1, and one step runs before the paired loop
    const bool odd = (nsteps & 1) != 0;
    char* first = odd ? st1 : st0;
    char* second = odd ? st0 : st1;
    dma(kb0, first);
    dma_wait();
    __syncthreads();
    if (nsteps > 1) dma(kb0 + 1, second);
    load_frag(f0, first, 0);
    if (nsteps == 1) {
        step_final(first);
    } else {
        int64_t s = 0;
        if (odd) {   // nsteps >= 3: block kb0 + 2 exists
            step_copy(st1, st0, kb0 + 2);
            s = 1;
        }
        // block kb0 + s is in st0 here
        for (; s + 3 < nsteps; s += 2) {
            step_copy(st0, st1, kb0 + s + 2);
            step_copy(st1, st0, kb0 + s + 3);
        }
        step_nocopy(st0, st1);
        step_final(st1);
    }

    if (splits == 1) {
        if (REQ)
            requant_tile<BIAS2, false>(acc, sAlpha, sBeta, M, N, m0, n0, wm, wn, lane, tid, nullptr, 0, st0, st1, ro);
        else
            store_tile<BIAS2, BN>(acc, sAlpha, sBeta, C, ldc, M, N, m0, n0, wm, wn, lane, false);
        return;
    }
    // K split in two: each half publishes its scaled values (C = ldexp(D, alpha_i + beta_j -
    // BIAS2), exact) in the tile's slot for that half and counts its arrival; the half that
    // arrives second adds the other's values to its own (the same fp32 sum as two atomic adds
    // into zero) and stores C.  Slot layout: thread t's acc[ti][tj] quarter q (four floats) at
    // ((((t / 64) * 16 + ti * 4 + tj) * 4 + q) * 1024 + (t % 64) * 16), coalesced 1 KB per store.
    // The slots are written and read with device-coherent accesses, so no cache write-back or
    // invalidation is needed: every thread waits for its stores to complete, the barrier orders
    // that before the arrival (a device-scope atomic), and the second half's reads are issued
    // only after it has seen the first half's arrival.
    const int64_t tile = (int64_t)wi.ty * RTB + wi.tx;
    char* slots = part + tile * 2 * PART_BYTES;
    const int wbase = (tid >> 6) * 16 * 4096 + lane * 16;
    {
        const int lcol = wn * WN + (lane & 31), lrow = wm * WM + 4 * (lane >> 5);
        const __amdgpu_buffer_rsrc_t rp = __builtin_amdgcn_make_buffer_rsrc(
            (void*)(slots + wi.split * PART_BYTES), (short)0, (int)PART_BYTES, 0x00020000);
#pragma unroll
        for (int ti = 0; ti < TM; ti++)
#pragma unroll
            for (int tj = 0; tj < TN; tj++) {
                const int beta = sBeta[lcol + 32 * tj] - BIAS2;
#pragma unroll
                for (int q = 0; q < 4; q++) {
                    const int4 al = *reinterpret_cast<const int4*>(sAlpha + lrow + 32 * ti + 8 * q);
                    f32x4 v;
                    v[0] = __builtin_amdgcn_ldexpf(acc[ti][tj][4 * q], al.x + beta);
                    v[1] = __builtin_amdgcn_ldexpf(acc[ti][tj][4 * q + 1], al.y + beta);
                    v[2] = __builtin_amdgcn_ldexpf(acc[ti][tj][4 * q + 2], al.z + beta);
                    v[3] = __builtin_amdgcn_ldexpf(acc[ti][tj][4 * q + 3], al.w + beta);
                    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), rp,
                                                           wbase + ((ti * 4 + tj) * 4 + q) * 1024, 0,
                                                           AUX_DEVICE_COHERENT);
                }
            }
    }
    __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0): this thread's slot stores are complete
    __syncthreads();
    if (tid == 0)
        sLast[0] = __hip_atomic_fetch_add(cnt + tile, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == 1;
    __syncthreads();
    if (!sLast[0]) return;   // uniform: the other half arrives later and finishes the tile
    if (REQ)
        requant_tile<BIAS2, true>(acc, sAlpha, sBeta, M, N, m0, n0, wm, wn, lane, tid,
                                  slots + (1 - wi.split) * PART_BYTES, wbase, st0, st1, ro);
    else
        store_tile<BIAS2, BN, true>(acc, sAlpha, sBeta, C, ldc, M, N, m0, n0, wm, wn, lane, false,
                                    slots + (1 - wi.split) * PART_BYTES, wbase);
}

// ---------------------------------------------------------------------------------------------
// Mixed formats and reused forward operands (the backward recipe of Sec. 3.3: E5C2 output
// gradients times the E4C3 codes kept from the forward pass).
//
// An operand is either the codes of an [R][K] tensor quantized along K (as above), or the codes
// of a [K][R] tensor quantized along R: a forward operand reused by a backward GEMM, whose
// block scales then run along the GEMM's rows, so the scale changes from element to element
// along k.  The expansion is the same but for the multiplier 2^-D, D = alpha_row - a, which is
// taken per element; the planes, and so the GEMM kernel, do not change.  Two formats need
// nothing else: each operand goes through its own format's table, the matrix cores multiply
// the values (the lift of both curve indices to the finer lattice is implicit in the values),
// and the epilogue removes the sum of the two operands' exponent offsets.
//
// Workspace: the single-format layout, then per operand the partial column maxima of a
// [K][R/32] scale matrix over slabs of 256 k-rows, [ceil(K/256)][RT * 8] int32.
constexpr int PREP_SLAB = 256;

struct MixedLayout {
    WsLayout w;
    int64_t nslab, colpart_a, colpart_b, bytes;
};

MixedLayout mixed_layout(int64_t M, int64_t N, int64_t K) {
    MixedLayout x;
    x.w = ws_layout(M, N, K);
    x.nslab = (K + PREP_SLAB - 1) / PREP_SLAB;
    x.colpart_a = (x.w.bytes + 255) & ~(int64_t)255;
    x.colpart_b = x.colpart_a + ((x.nslab * x.w.rta * 8 * 4 + 255) & ~(int64_t)255);
    x.bytes = x.colpart_b + x.nslab * x.w.rtb * 8 * 4;
    return x;
}

struct PrepOperand {
    const int8_t* scales;
    int64_t rows, tiles, K;
    int trans;
    int groups;     // workgroups of this operand
    int cgroups;    // trans: groups of 64 scale columns covering the tiles' tiles * 8 columns
    int* rmax;      // not trans: row maxima [tiles * 256], 0 past the last row
    int* colpart;   // trans: partial column maxima [nslab][tiles * 8]
    int64_t nsb;    // scales per row (not trans: K / G) or per k-row (trans: rows / G)
    Div32 dgq;      // trans: 32-row group j has scale column j / (G / 32)
};

// one launch before the expansion: for an operand quantized along K, the row maxima of its block
// scales (16 lanes per row, as prep_kernel); for a reused operand, the maxima of each scale
// column over a slab of 256 k-rows (64 columns x 4 parts of 64 k-rows per workgroup, a wave
// reading 64 consecutive scale bytes of one k-row).  One more workgroup zeroes the per-tile
// arrival counters when K is split.
__global__ __launch_bounds__(256) void prep_mixed_kernel(PrepOperand pa, PrepOperand pb, int* __restrict__ cnt,
                                                         int ncnt) {
    __shared__ int red[256];
    const int bid = (int)blockIdx.x, t = (int)threadIdx.x;
    if (bid >= pa.groups + pb.groups) {
        for (int i = t; i < ncnt; i += 256) cnt[i] = 0;
        return;
    }
    const bool isA = bid < pa.groups;
    const PrepOperand& p = isA ? pa : pb;
    const int g = isA ? bid : bid - pa.groups;
    if (!p.trans) {
        const int64_t nsb = p.nsb;
        const int64_t row = (int64_t)g * 16 + (t >> 4);
        const int part = t & 15;
        int m = -128;
        if (row < p.rows) {
            const int8_t* sp = p.scales + row * nsb;
#pragma unroll 8
            for (int64_t sb = part; sb < nsb; sb += 16) m = max(m, scale_key((int)sp[sb]));
        }
#pragma unroll
        for (int o = 8; o > 0; o >>= 1) m = max(m, __shfl_xor(m, o, 16));
        if (part == 0) p.rmax[row] = row < p.rows ? m : 0;   // the grid covers exactly the padded rows
        return;
    }
    const int64_t J = p.rows / 32, J8 = p.tiles * 8;
    const int cg = g % p.cgroups, slab = g / p.cgroups;
    const int64_t j = (int64_t)cg * 64 + (t & 63);
    const int64_t k0 = (int64_t)slab * PREP_SLAB + (t >> 6) * 64;
    int m = -128;
    if (j < J) {
        const int8_t* sp = p.scales + div32((uint32_t)j, p.dgq);
        const int64_t kend = min(k0 + 64, p.K);
#pragma unroll 8
        for (int64_t k = k0; k < kend; k++) m = max(m, scale_key((int)sp[k * p.nsb]));
    }
    red[t] = m;
    __syncthreads();
    if (t < 64 && j < J8)
        p.colpart[(int64_t)slab * J8 + j] = max(max(red[t], red[t + 64]), max(red[t + 128], red[t + 192]));
}

struct ExpandTOperand {
    const uint8_t* codes;    // [K][ld] bytes: codes of a [K][R] tensor quantized along R
    const int8_t* scales;    // [K][R / G]
    int64_t rows, tiles, ld; // R, row tiles of 256, bytes per k-row (R, or R / 32 * 28 packed)
    const int* colpart;      // partial column maxima [nslab][tiles * 8]
    int64_t nslab;
    int* rmax;               // row maxima [tiles * 256], written by the first K block's workgroups
    char* planes;
    int fidx;
    int64_t nsb;             // scales per k-row, R / G
    Div32 dgq;               // 32-row group j has scale column j / (G / 32)
};

// expansion of a reused operand: one workgroup per (K block, tile of 256 rows).  The 32 k-rows
// x 256 codes are read with coalesced dword loads into LDS (pitch one dword over the row, so the
// four 8-wide k-chunks a wave reads fall on different banks), the block scales transposed into
// [8 scale columns][32 k].  Thread t then writes chunk q = t % 4 (k = 8q .. 8q + 7) of rows
// t / 4 + 64 i, i < 4, into both planes: each store of a wave covers 16 whole 64-byte rows.
// Every element is scaled by 2^-min(D, 24) and then by 2^-min(max(D - 24, 0), 24) (a multiply
// by one when D <= 24), the two multiplies of the K-layout expansion with D taken per element.
template <bool P7>
__global__ __launch_bounds__(256) void expand_t_kernel(ExpandTOperand opA, ExpandTOperand opB) {
    constexpr int TB = P7 ? 224 : 256;   // code bytes of one k-row of a 256-row tile
    constexpr int DPR = TB / 4;          // dwords per k-row
    constexpr int PITCH = DPR + 1;
    __shared__ uint32_t lut[GEMM_DEC_ENTRIES];
    __shared__ uint32_t tile[32 * PITCH];
    __shared__ __attribute__((aligned(16))) int8_t scT[8 * 32];
    __shared__ int alpha_s[8];
    const int t = (int)threadIdx.x;
    const bool isA = (int64_t)blockIdx.y < opA.tiles;
    const ExpandTOperand& op = isA ? opA : opB;
    lut[t] = g_dec[op.fidx][t];
    const int64_t rt = isA ? (int64_t)blockIdx.y : (int64_t)blockIdx.y - opA.tiles;
    const int64_t kb = blockIdx.x;
    const int64_t R = op.rows, J8 = op.tiles * 8;
    const int vrows = (int)min((int64_t)256, R - rt * 256);   // a multiple of 32
    const int vdw = P7 ? vrows / 32 * 7 : vrows / 4;           // valid dwords of a k-row
    const uint8_t* src = op.codes + kb * 32 * op.ld + rt * TB;
#pragma unroll
    for (int i = 0; i < 32 * DPR / 256; i++) {
        const int d = t + 256 * i;
        const int k = d / DPR, c = d - k * DPR;
        uint32_t v = 0;
        if (c < vdw) v = *reinterpret_cast<const uint32_t*>(src + k * op.ld + 4 * c);
        tile[k * PITCH + c] = v;
    }
    {
        const int k = t >> 3, j = t & 7;
        int s = -128;
        if (32 * j < vrows) s = op.scales[(kb * 32 + k) * op.nsb + div32((uint32_t)(rt * 8 + j), op.dgq)];
        scT[j * 32 + k] = (int8_t)s;
    }
    {
        // the row maxima of this tile's 8 scale columns, finished from the slab partials
        const int j = t >> 5, l = t & 31;
        int m = -128;
        for (int64_t sl = l; sl < op.nslab; sl += 32) m = max(m, op.colpart[sl * J8 + rt * 8 + j]);
#pragma unroll
        for (int o = 16; o > 0; o >>= 1) m = max(m, __shfl_xor(m, o, 32));
        if (l == 0) alpha_s[j] = 32 * j < vrows ? m : 0;
    }
    __syncthreads();
    if (kb == 0) op.rmax[rt * 256 + t] = alpha_s[t >> 5];
    const int q = t & 3, rb = t >> 2;
    const uint8_t* tb = reinterpret_cast<const uint8_t*>(tile);
    char* base = op.planes + (kb * op.tiles + rt) * (2 * PLANE);
#pragma unroll
    for (int i = 0; i < 4; i++) {
        const int r = rb + 64 * i, j = r >> 5;
        const int alpha = alpha_s[j];
        const uint2 sv = *reinterpret_cast<const uint2*>(scT + j * 32 + 8 * q);
        uint32_t e[8], m1[8], m2[8];
#pragma unroll
        for (int x = 0; x < 8; x++) {
            const int k = 8 * q + x;
            uint32_t code;
            if (!P7) {
                code = tb[k * PITCH * 4 + r];
            } else {
                const int bit = 224 * j + 7 * (r & 31);
                const int byte = k * PITCH * 4 + (bit >> 3);
                code = ((uint32_t)tb[byte] | ((uint32_t)tb[byte + 1] << 8)) >> (bit & 7) & 0x7Fu;
            }
            e[x] = lut[code];
            const int a = (int)__builtin_amdgcn_sbfe(x < 4 ? sv.x : sv.y, 8 * (x & 3), 8);
            const int D = alpha - a;
            m1[x] = f16_pow2_neg(min(max(D, 0), 24));
            m2[x] = f16_pow2_neg(min(max(D - 24, 0), 24));
        }
        uint32_t hv[4], lv[4];
#pragma unroll
        for (int p = 0; p < 4; p++) {
            const half2v s1 = __builtin_bit_cast(half2v, m1[2 * p] | (m1[2 * p + 1] << 16));
            const half2v s2 = __builtin_bit_cast(half2v, m2[2 * p] | (m2[2 * p + 1] << 16));
            hv[p] = pk_mul(pk_mul(__builtin_amdgcn_perm(e[2 * p + 1], e[2 * p], 0x05040100u), s1), s2);
            lv[p] = pk_mul(pk_mul(__builtin_amdgcn_perm(e[2 * p + 1], e[2 * p], 0x07060302u), s1), s2);
        }
        char* dst = base + swz(r, q);
        *reinterpret_cast<uint4*>(dst) = make_uint4(hv[0], hv[1], hv[2], hv[3]);
        *reinterpret_cast<uint4*>(dst + PLANE) = make_uint4(lv[0], lv[1], lv[2], lv[3]);
    }
}

template <class F>
hipError_t launch_ws_fmt(const void* a, const int8_t* as, const void* b, const int8_t* bs, int64_t M,
                         int64_t N, int64_t K, int block, float* c, int64_t ldc, char* ws, int fidx, hipStream_t s) {
    hipError_t e = hipSuccess;
    const WsLayout w = ws_layout(M, N, K);
    const int64_t nkb = K / 32, nsb = K / block;
    const Div32 dgq = make_div32((uint32_t)(block / 32));
    int* maxA = reinterpret_cast<int*>(ws + w.max_a);
    int* maxB = reinterpret_cast<int*>(ws + w.max_b);
    const int64_t tiles = w.rta * w.rtb;
    const int splits = w.splits;
    int* cnt = reinterpret_cast<int*>(ws + w.cnt);
    const int ga = (int)(w.rta * BM / 16), gb = (int)(w.rtb * BM / 16);
    const int ncnt = splits > 1 ? (int)tiles : 0;
    hipLaunchKernelGGL(prep_kernel, dim3((unsigned)(ga + gb + (splits > 1 ? 1 : 0))), dim3(256), 0, s, as, bs, M, N,
                       nsb, ga, gb, maxA, maxB, cnt, ncnt);
    const ExpandOperand opA = {reinterpret_cast<const uint8_t*>(a), as, M, w.rta, maxA, ws + w.planes_a, fidx, nsb, dgq};
    const ExpandOperand opB = {reinterpret_cast<const uint8_t*>(b), bs, N, w.rtb, maxB, ws + w.planes_b, fidx, nsb, dgq};
    hipLaunchKernelGGL((expand_kernel<F>), dim3((unsigned)(4 * (w.rta + w.rtb)), (unsigned)((nkb + 3) / 4)),
                       dim3(256), 0, s, opA, opB, nkb);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int64_t items = w.rta * w.rtb * splits;
    const int64_t grid = (items + 7) / 8 * 8;   // whole XCD shares; surplus workgroups return at once
    hipLaunchKernelGGL((gemm_ws_kernel<2 * F::GEMM_BIAS>), dim3((unsigned)grid), dim3(NTHREADS), 0, s, ws + w.planes_a,
                       ws + w.planes_b, maxA, maxB, M, N, K, w.rta, w.rtb, c, ldc, splits, ws + w.part, cnt, ReqOut{});
    return hipGetLastError();
}

// curvefp_gemm_ws with its epilogue requantizing C (see requant_tile): the same prep and
// expansion launches, then gemm_ws_kernel<BIAS2, true>
template <class F>
hipError_t launch_requant_fmt(const void* a, const int8_t* as, const void* b, const int8_t* bs, int64_t M,
                              int64_t N, int64_t K, int block, char* ws, int fidx, int ofmt, int oblock, uint8_t* qc,
                              int8_t* qs, hipStream_t s) {
    const WsLayout w = ws_layout(M, N, K);
    const int64_t nkb = K / 32, nsb = K / block;
    const Div32 dgq = make_div32((uint32_t)(block / 32));
    int* maxA = reinterpret_cast<int*>(ws + w.max_a);
    int* maxB = reinterpret_cast<int*>(ws + w.max_b);
    const int64_t tiles = w.rta * w.rtb;
    const int splits = w.splits;
    int* cnt = reinterpret_cast<int*>(ws + w.cnt);
    const int ga = (int)(w.rta * BM / 16), gb = (int)(w.rtb * BM / 16);
    const int ncnt = splits > 1 ? (int)tiles : 0;
    hipLaunchKernelGGL(prep_kernel, dim3((unsigned)(ga + gb + (splits > 1 ? 1 : 0))), dim3(256), 0, s, as, bs, M, N,
                       nsb, ga, gb, maxA, maxB, cnt, ncnt);
    const ExpandOperand opA = {reinterpret_cast<const uint8_t*>(a), as, M, w.rta, maxA, ws + w.planes_a, fidx, nsb, dgq};
    const ExpandOperand opB = {reinterpret_cast<const uint8_t*>(b), bs, N, w.rtb, maxB, ws + w.planes_b, fidx, nsb, dgq};
    hipLaunchKernelGGL((expand_kernel<F>), dim3((unsigned)(4 * (w.rta + w.rtb)), (unsigned)((nkb + 3) / 4)),
                       dim3(256), 0, s, opA, opB, nkb);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    int glog = 0;
    while ((32 << glog) < oblock) glog++;
    const ReqOut ro{qc, qs, qrule(ofmt), ofmt, ofmt == 2 ? 1 : 0, glog};
    const int64_t grid = (tiles * splits + 7) / 8 * 8;
    hipLaunchKernelGGL((gemm_ws_kernel<2 * F::GEMM_BIAS, true>), dim3((unsigned)grid), dim3(NTHREADS), 0, s,
                       ws + w.planes_a, ws + w.planes_b, maxA, maxB, M, N, K, w.rta, w.rtb, nullptr, N, splits,
                       ws + w.part, cnt, ro);
    return hipGetLastError();
}

// fp16 exponent offset of a format's expansion (the row's largest element lands near 2^15)
int gemm_bias(int f) {
    constexpr int bias[NUM_FORMATS] = {FmtE4C3::GEMM_BIAS, FmtE5C2::GEMM_BIAS, FmtE3C3::GEMM_BIAS,
                                       FmtE4C3R89::GEMM_BIAS, FmtE4C3R34::GEMM_BIAS};
    return bias[f];
}

// the GEMM kernel for the sum of the two operands' offsets: E4C3 and 2^(8/9) 8, E5C2 0, E3C3 12,
// 2^(3/4) 10, so the sums of any two are 0, 8, 10, 12, 16, 18, 20, 22, 24
hipError_t launch_gemm_ws_bias(int bias2, dim3 grid, hipStream_t s, const char* pa, const char* pb, const int* maxA,
                               const int* maxB, int64_t M, int64_t N, int64_t K, int64_t rta, int64_t rtb, float* c,
                               int64_t ldc, int splits, char* part, int* cnt) {
    static_assert(FmtE4C3::GEMM_BIAS == 8 && FmtE5C2::GEMM_BIAS == 0 && FmtE3C3::GEMM_BIAS == 12 &&
                      FmtE4C3R89::GEMM_BIAS == 8 && FmtE4C3R34::GEMM_BIAS == 10,
                  "the bias sums listed below");
#define CURVEFP_WS_GEMM(B2)                                                                                     \
    case B2:                                                                                                  \
        hipLaunchKernelGGL((gemm_ws_kernel<B2>), grid, dim3(NTHREADS), 0, s, pa, pb, maxA, maxB, M, N, K, rta, \
                           rtb, c, ldc, splits, part, cnt, ReqOut{});                                         \
        break;
    switch (bias2) {
        CURVEFP_WS_GEMM(0)
        CURVEFP_WS_GEMM(8)
        CURVEFP_WS_GEMM(10)
        CURVEFP_WS_GEMM(12)
        CURVEFP_WS_GEMM(16)
        CURVEFP_WS_GEMM(18)
        CURVEFP_WS_GEMM(20)
        CURVEFP_WS_GEMM(22)
        CURVEFP_WS_GEMM(24)
        default: return hipErrorInvalidValue;
    }
#undef CURVEFP_WS_GEMM
    return hipGetLastError();
}

hipError_t launch_mixed(const void* a, const int8_t* as, int fa, int ta, const void* b, const int8_t* bs, int fb,
                        int tb, int64_t M, int64_t N, int64_t K, int block, float* c, int64_t ldc, char* ws,
                        hipStream_t s) {
    const MixedLayout x = mixed_layout(M, N, K);
    const WsLayout& w = x.w;
    const int64_t nkb = K / 32;
    const Div32 dgq = make_div32((uint32_t)(block / 32));
    int* maxA = reinterpret_cast<int*>(ws + w.max_a);
    int* maxB = reinterpret_cast<int*>(ws + w.max_b);
    int* cnt = reinterpret_cast<int*>(ws + w.cnt);
    const int64_t tiles = w.rta * w.rtb;
    const int splits = w.splits;
    auto prep_op = [&](const int8_t* sc, int64_t R, int64_t RT, int tr, int* rmax, int64_t colpart) {
        PrepOperand p;
        p.scales = sc;
        p.rows = R;
        p.tiles = RT;
        p.K = K;
        p.trans = tr;
        p.cgroups = (int)((RT * 8 + 63) / 64);
        p.groups = tr ? (int)(p.cgroups * x.nslab) : (int)(RT * 16);
        p.rmax = rmax;
        p.colpart = reinterpret_cast<int*>(ws + colpart);
        p.nsb = tr ? R / block : K / block;
        p.dgq = dgq;
        return p;
    };
    const PrepOperand pa = prep_op(as, M, w.rta, ta, maxA, x.colpart_a);
    const PrepOperand pb = prep_op(bs, N, w.rtb, tb, maxB, x.colpart_b);
    hipLaunchKernelGGL(prep_mixed_kernel, dim3((unsigned)(pa.groups + pb.groups + (splits > 1 ? 1 : 0))), dim3(256), 0,
                       s, pa, pb, cnt, (int)(splits > 1 ? tiles : 0));
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;

    // expansions: operands that share a kind (along K, or reused) and a code packing share a launch
    const bool p7a = fa == 2, p7b = fb == 2;
    const int64_t nsb = K / block;
    const ExpandOperand ka = {reinterpret_cast<const uint8_t*>(a), as, M, w.rta, maxA, ws + w.planes_a, fa, nsb, dgq};
    const ExpandOperand kbo = {reinterpret_cast<const uint8_t*>(b), bs, N, w.rtb, maxB, ws + w.planes_b, fb, nsb, dgq};
    auto ld_of = [](int f, int64_t R) { return f == 2 ? R / 32 * 28 : R; };
    const ExpandTOperand xa = {reinterpret_cast<const uint8_t*>(a), as, M, w.rta, ld_of(fa, M),
                               reinterpret_cast<const int*>(ws + x.colpart_a), x.nslab, maxA, ws + w.planes_a, fa,
                               M / block, dgq};
    const ExpandTOperand xb = {reinterpret_cast<const uint8_t*>(b), bs, N, w.rtb, ld_of(fb, N),
                               reinterpret_cast<const int*>(ws + x.colpart_b), x.nslab, maxB, ws + w.planes_b, fb,
                               N / block, dgq};
    auto expand_k = [&](const ExpandOperand& o1, const ExpandOperand& o2, bool p7) {
        const dim3 grid((unsigned)(4 * (o1.tiles + o2.tiles)), (unsigned)((nkb + 3) / 4));
        if (p7) hipLaunchKernelGGL((expand_kernel<FmtE3C3>), grid, dim3(256), 0, s, o1, o2, nkb);
        else hipLaunchKernelGGL((expand_kernel<FmtE4C3>), grid, dim3(256), 0, s, o1, o2, nkb);
        return hipGetLastError();
    };
    auto expand_t = [&](const ExpandTOperand& o1, const ExpandTOperand& o2, bool p7) {
        const dim3 grid((unsigned)nkb, (unsigned)(o1.tiles + o2.tiles));
        if (p7) hipLaunchKernelGGL((expand_t_kernel<true>), grid, dim3(256), 0, s, o1, o2);
        else hipLaunchKernelGGL((expand_t_kernel<false>), grid, dim3(256), 0, s, o1, o2);
        return hipGetLastError();
    };
    ExpandOperand kn = ka;
    kn.tiles = 0;   // an absent second operand: no workgroups
    ExpandTOperand xn = xa;
    xn.tiles = 0;
    if (ta == tb && p7a == p7b) {
        e = ta ? expand_t(xa, xb, p7a) : expand_k(ka, kbo, p7a);
    } else {
        e = ta ? expand_t(xa, xn, p7a) : expand_k(ka, kn, p7a);
        if (e == hipSuccess) e = tb ? expand_t(xb, xn, p7b) : expand_k(kbo, kn, p7b);
    }
    if (e != hipSuccess) return e;
    const int64_t items = tiles * splits;
    const dim3 grid((unsigned)((items + 7) / 8 * 8));
    return launch_gemm_ws_bias(gemm_bias(fa) + gemm_bias(fb), grid, s, ws + w.planes_a, ws + w.planes_b, maxA, maxB,
                               M, N, K, w.rta, w.rtb, c, ldc, splits, ws + w.part, cnt);
}

template <class F, int BN_>
hipError_t launch_tile(const void* a, const int8_t* as, const void* b, const int8_t* bs, int64_t M,
                       int64_t N, int64_t K, int block, float* c, int64_t ldc, int fidx, int splits, hipStream_t s) {
    hipError_t e = hipSuccess;
    if (splits > 1) {
        int64_t zb = (M * N + 255) / 256;
        zb = zb < 4096 ? zb : 4096;
        hipLaunchKernelGGL(zero_rows_kernel, dim3((unsigned)zb), dim3(256), 0, s, c, M, N, ldc);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    dim3 grid((unsigned)((N + BN_ - 1) / BN_), (unsigned)((M + BM - 1) / BM), (unsigned)splits);
    hipLaunchKernelGGL((gemm_kernel<F, BN_>), grid, dim3(NTHREADS), 0, s,
                       reinterpret_cast<const uint8_t*>(a), as, reinterpret_cast<const uint8_t*>(b), bs,
                       M, N, K, c, ldc, fidx, K / block, make_div32((uint32_t)(block / 32)));
    return hipGetLastError();
}

// 256 x 256 tiles; K is split in two (partial sums added into a cleared C) when the tiles cover
// fewer than the 256 compute units and K is long enough.  (256 x 128 tiles without a split
// measured 17% slower on 2048 x 4096 x 4096.)
template <class F>
hipError_t launch_fmt(const void* a, const int8_t* as, const void* b, const int8_t* bs, int64_t M,
                      int64_t N, int64_t K, int block, float* c, int64_t ldc, int fidx, hipStream_t s) {
    const int64_t tiles = ((M + BM - 1) / BM) * ((N + 255) / 256);
    const int splits = (tiles < 256 && K / 32 >= 16) ? 2 : 1;
    return launch_tile<F, 256>(a, as, b, bs, M, N, K, block, c, ldc, fidx, splits, s);
}

// Prepared operands: one operand's expansion in a buffer of its own, so that an operand several
// GEMMs share (static weights) is expanded once, and the two operands can be expanded on two
// streams as soon as each is quantized.  Layout for [rows][K] codes quantized along K: the planes
// [K/32][RT][hi, lo][256 rows][64 B] (RT = ceil(rows / 256)), exactly the workspace path's
// planes of that operand, then the row maxima of its block scales (prep_kernel's keys), RT * 256
// int32.  A reused operand (codes of a [K][rows] tensor quantized along rows, the backward GEMMs'
// forward operand) is expanded into the same planes and row maxima, followed by the partial column
// maxima its expansion reads ([ceil(K / 256)][RT * 8] int32, scratch of the preparation).  The
// expansion depends on the operand alone, so prepare(A), prepare(B) and gemm_prepared give
// curvefp_gemm_ws's C (and curvefp_gemm_mixed's, for two formats or reused operands) bit for bit.
struct PreparedLayout {
    int64_t rt, planes, rmax, colpart, nslab, bytes;
};

PreparedLayout prepared_layout(int64_t rows, int64_t K, int trans = 0) {
    PreparedLayout p;
    p.rt = (rows + BM - 1) / BM;
    p.planes = 0;
    p.rmax = (K / 32) * p.rt * 2 * PLANE;
    p.bytes = p.rmax + p.rt * BM * 4;
    p.nslab = (K + PREP_SLAB - 1) / PREP_SLAB;
    p.colpart = p.bytes;
    if (trans) p.bytes = p.colpart + p.nslab * p.rt * 8 * 4;
    return p;
}

// the workspace of a GEMM on prepared operands: nothing unless K is split (then the arrival
// counters and partial-sum slots of the workspace path)
struct PreparedGemmLayout {
    int64_t cnt, part, bytes;
    int splits;
};

PreparedGemmLayout prepared_gemm_layout(int64_t M, int64_t N, int64_t K) {
    const WsLayout w = ws_layout(M, N, K);
    PreparedGemmLayout g;
    g.splits = w.splits;
    g.cnt = g.part = g.bytes = 0;
    if (g.splits > 1) {
        const int64_t tiles = w.rta * w.rtb;
        g.part = (tiles * 4 + 255) & ~(int64_t)255;
        g.bytes = g.part + tiles * g.splits * PART_BYTES;
    }
    return g;
}

}  // namespace

int64_t gemm_workspace_bytes(int64_t M, int64_t N, int64_t K) { return ws_layout(M, N, K).bytes; }

int64_t prepared_bytes(int64_t rows, int64_t K, int trans) { return prepared_layout(rows, K, trans).bytes; }

int64_t gemm_prepared_workspace_bytes(int64_t M, int64_t N, int64_t K) { return prepared_gemm_layout(M, N, K).bytes; }

hipError_t launch_prepare(const void* codes, const int8_t* scales, int64_t rows, int64_t K, int format, int block,
                          int trans, void* prepared, hipStream_t s) {
    const PreparedLayout p = prepared_layout(rows, K, trans);
    const int64_t nkb = K / 32, nsb = K / block;
    char* base = reinterpret_cast<char*>(prepared);
    int* rmax = reinterpret_cast<int*>(base + p.rmax);
    if (trans) {
        // the mixed path's preparation of a reused operand: partial column maxima of its scales
        // over slabs of 256 k-rows (prep_mixed_kernel), then the transposed expansion, which
        // takes each row's maximum from them and writes it beside the planes
        const Div32 dgq = make_div32((uint32_t)(block / 32));
        PrepOperand po;
        po.scales = scales;
        po.rows = rows;
        po.tiles = p.rt;
        po.K = K;
        po.trans = 1;
        po.cgroups = (int)((p.rt * 8 + 63) / 64);
        po.groups = (int)(po.cgroups * p.nslab);
        po.rmax = rmax;
        po.colpart = reinterpret_cast<int*>(base + p.colpart);
        po.nsb = rows / block;
        po.dgq = dgq;
        PrepOperand pn = po;
        pn.groups = 0;   // no second operand
        hipLaunchKernelGGL(prep_mixed_kernel, dim3((unsigned)po.groups), dim3(256), 0, s, po, pn, (int*)nullptr, 0);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        const ExpandTOperand xo = {reinterpret_cast<const uint8_t*>(codes), scales, rows, p.rt,
                                   format == 2 ? rows / 32 * 28 : rows, po.colpart, p.nslab, rmax, base + p.planes,
                                   format, rows / block, dgq};
        ExpandTOperand xn = xo;
        xn.tiles = 0;
        const dim3 grid((unsigned)nkb, (unsigned)p.rt);
        if (format == 2) hipLaunchKernelGGL((expand_t_kernel<true>), grid, dim3(256), 0, s, xo, xn);
        else hipLaunchKernelGGL((expand_t_kernel<false>), grid, dim3(256), 0, s, xo, xn);
        return hipGetLastError();
    }
    const int groups = (int)(p.rt * BM / 16);
    hipLaunchKernelGGL(prep_kernel, dim3((unsigned)groups), dim3(256), 0, s, scales, (const int8_t*)nullptr, rows,
                       (int64_t)0, nsb, groups, 0, rmax, (int*)nullptr, (int*)nullptr, 0);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const ExpandOperand op = {reinterpret_cast<const uint8_t*>(codes), scales, rows, p.rt, rmax, base + p.planes,
                              format, nsb, make_div32((uint32_t)(block / 32))};
    ExpandOperand none = op;
    none.tiles = 0;   // no second operand: no workgroups
    // the kernel's format parameter fixes only the code packing; the table is the operand's
    const dim3 grid((unsigned)(4 * p.rt), (unsigned)((nkb + 3) / 4));
    if (format == 2) hipLaunchKernelGGL((expand_kernel<FmtE3C3>), grid, dim3(256), 0, s, op, none, nkb);
    else hipLaunchKernelGGL((expand_kernel<FmtE4C3>), grid, dim3(256), 0, s, op, none, nkb);
    return hipGetLastError();
}

hipError_t launch_gemm_prepared(const void* pa, int fa, const void* pb, int fb, int64_t M, int64_t N, int64_t K,
                                float* c, int64_t ldc, void* ws, hipStream_t s) {
    const PreparedLayout la = prepared_layout(M, K), lb = prepared_layout(N, K);
    const PreparedGemmLayout g = prepared_gemm_layout(M, N, K);
    const char* a = reinterpret_cast<const char*>(pa);
    const char* b = reinterpret_cast<const char*>(pb);
    const int64_t tiles = la.rt * lb.rt;
    char* w = reinterpret_cast<char*>(ws);
    int* cnt = g.splits > 1 ? reinterpret_cast<int*>(w + g.cnt) : nullptr;
    if (g.splits > 1) {
        // prep_kernel with no operands: its one extra workgroup clears the arrival counters
        hipLaunchKernelGGL(prep_kernel, dim3(1), dim3(256), 0, s, (const int8_t*)nullptr, (const int8_t*)nullptr,
                           (int64_t)0, (int64_t)0, (int64_t)0, 0, 0, (int*)nullptr, (int*)nullptr, cnt, (int)tiles);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    const int64_t items = tiles * g.splits;
    const dim3 grid((unsigned)((items + 7) / 8 * 8));
    return launch_gemm_ws_bias(gemm_bias(fa) + gemm_bias(fb), grid, s, a + la.planes, b + lb.planes,
                               reinterpret_cast<const int*>(a + la.rmax), reinterpret_cast<const int*>(b + lb.rmax),
                               M, N, K, la.rt, lb.rt, c, ldc, g.splits, g.splits > 1 ? w + g.part : nullptr, cnt);
}

int64_t gemm_mixed_workspace_bytes(int64_t M, int64_t N, int64_t K) { return mixed_layout(M, N, K).bytes; }

hipError_t launch_gemm_requant(const void* a, const int8_t* as, const void* b, const int8_t* bs, int64_t M, int64_t N,
                               int64_t K, int format, int block, int out_format, int out_block, void* out_codes,
                               int8_t* out_scales, void* ws, hipStream_t s) {
    char* w = reinterpret_cast<char*>(ws);
    uint8_t* qc = reinterpret_cast<uint8_t*>(out_codes);
    switch (format) {
        case 0: return launch_requant_fmt<FmtE4C3>(a, as, b, bs, M, N, K, block, w, 0, out_format, out_block, qc, out_scales, s);
        case 1: return launch_requant_fmt<FmtE5C2>(a, as, b, bs, M, N, K, block, w, 1, out_format, out_block, qc, out_scales, s);
        case 2: return launch_requant_fmt<FmtE3C3>(a, as, b, bs, M, N, K, block, w, 2, out_format, out_block, qc, out_scales, s);
        case 3: return launch_requant_fmt<FmtE4C3>(a, as, b, bs, M, N, K, block, w, 3, out_format, out_block, qc, out_scales, s);
        default: return launch_requant_fmt<FmtE4C3R34>(a, as, b, bs, M, N, K, block, w, 4, out_format, out_block, qc, out_scales, s);
    }
}

hipError_t launch_gemm_mixed(const void* a, const int8_t* as, int fa, int ta, const void* b, const int8_t* bs, int fb,
                             int tb, int64_t M, int64_t N, int64_t K, int block, float* c, int64_t ldc, void* ws,
                             hipStream_t s) {
    return launch_mixed(a, as, fa, ta, b, bs, fb, tb, M, N, K, block, c, ldc, reinterpret_cast<char*>(ws), s);
}

hipError_t launch_gemm_ws(const void* a, const int8_t* as, const void* b, const int8_t* bs, int64_t M,
                          int64_t N, int64_t K, int format, int block, float* c, int64_t ldc, void* ws,
                          hipStream_t s) {
    char* w = reinterpret_cast<char*>(ws);
    switch (format) {
        case 0: return launch_ws_fmt<FmtE4C3>(a, as, b, bs, M, N, K, block, c, ldc, w, 0, s);
        case 1: return launch_ws_fmt<FmtE5C2>(a, as, b, bs, M, N, K, block, c, ldc, w, 1, s);
        case 2: return launch_ws_fmt<FmtE3C3>(a, as, b, bs, M, N, K, block, c, ldc, w, 2, s);
        // 2^(8/9) shares E4C3's packing and exponent offset: its kernels, its own table
        case 3: return launch_ws_fmt<FmtE4C3>(a, as, b, bs, M, N, K, block, c, ldc, w, 3, s);
        default: return launch_ws_fmt<FmtE4C3R34>(a, as, b, bs, M, N, K, block, c, ldc, w, 4, s);
    }
}

hipError_t launch_gemm(const void* a, const int8_t* as, const void* b, const int8_t* bs, int64_t M,
                       int64_t N, int64_t K, int format, int block, float* c, int64_t ldc, hipStream_t s) {
    switch (format) {
        case 0: return launch_fmt<FmtE4C3>(a, as, b, bs, M, N, K, block, c, ldc, 0, s);
        case 1: return launch_fmt<FmtE5C2>(a, as, b, bs, M, N, K, block, c, ldc, 1, s);
        case 2: return launch_fmt<FmtE3C3>(a, as, b, bs, M, N, K, block, c, ldc, 2, s);
        case 3: return launch_fmt<FmtE4C3>(a, as, b, bs, M, N, K, block, c, ldc, 3, s);
        default: return launch_fmt<FmtE4C3R34>(a, as, b, bs, M, N, K, block, c, ldc, 4, s);
    }
}

}  // namespace curvefp
