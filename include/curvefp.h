/*
 * curvefp.h -- C ABI of libcurvefp: CurveFP block quantization, reconstruction
 * and the CurveFP GEMM on AMD Instinct MI355X (gfx950).
 *
 * CurveFP (arXiv 2608.10010) stores a block of G values with one signed
 * power-of-two scale exponent a_b and one (1+E+C)-bit code per element; a
 * nonzero element is (-1)^s 2^{a_b} r^{e + k/K}, K = 2^C (Sec. 3.1,
 * Eq. curvefp-value).  The formats are those of Tab. curvefp-formats:
 * CurveFP8 E4C3 (forward operands), CurveFP8 E5C2 (gradients) and CurveFP7
 * E3C3 (compact inference), all with binary radix r = 2, and E4C3 with the
 * radices r = 2^{8/9} and r = 2^{3/4} of Tab. radix-frontier.
 *
 * Conventions shared by every entry point
 *   - All data pointers are device pointers owned by the caller.  The library
 *     never allocates, frees or keeps them.
 *   - `stream` is a hipStream_t (NULL = the legacy default stream).  Every call
 *     is asynchronous on that stream and never synchronizes it.  The library
 *     keeps no state: its constant tables (quantizer thresholds, reconstruction
 *     and expansion values) are compile-time __constant__ arrays, generated
 *     when the library is built, so no call uploads, allocates or waits, and
 *     every call may be captured into a HIP graph.
 *   - Argument errors are detected before any HIP call and returned as a
 *     negative curvefp_status; nothing is launched then.  Launch failures
 *     return CURVEFP_ERR_HIP.  Data-dependent conditions (non-finite inputs)
 *     are encoded in the outputs, never in the status.
 *   - block G is the number of consecutive elements along the blocked axis that
 *     share one scale (Eq. effective-rate: R = 1 + E + C + S/G bits per value;
 *     Sec. 3.1 evaluates fixed-size blocks, rowwise and tensorwise sharing):
 *     any positive multiple of 32 (32, 64, ..., 512 for the block sizes the
 *     paper sweeps; the blocked extent itself for rowwise scales), else
 *     CURVEFP_ERR_BLOCK.  The blocked extent must be a multiple of G
 *     (CURVEFP_ERR_SHAPE otherwise).  curvefp_gemm_requant's output blocks are
 *     chosen on their own (32, 64, 128 or 256).
 *   - Code, output and (for blocks along rows) source pointers must be 16-byte
 *     aligned, and leading dimensions (in elements) must keep every row 16-byte
 *     aligned; the quantize-transpose source only needs element alignment.
 *
 * Element code layout (one byte per code for E4C3/E5C2, 7-bit packed for E3C3)
 *   code = s << (E+C) | m,  m = n + 2^{E+C-1},  n = e*K + k in [-(2^{E+C-1}-1), 2^{E+C-1}-1],
 *   standing for r^{n/K} = 2^{p n / (qK)},
 *   m = 0 is the zero sentinel (the paper reserves magnitude index zero and drops
 *   the smallest exponent/curve combination, Sec. 3.1; App. C.1 gives the same
 *   rank layout for E4C3: sign in bit 7, rank in bits 6:0, q = m - 64).
 *   Codes are laid out per group of 32 elements whatever G is.  E3C3 codes are
 *   packed LSB first: code i of a group of 32 occupies bits [7i, 7i+7) of a
 *   224-bit little-endian string, i.e. 28 bytes per group.
 *
 * Scales: int8 power-of-two exponents, one per block of G, row-major
 *   [outer][k / G]; -128 marks a block that held a NaN or an infinity.  A block's
 *   scale is the ceil-absmax rule applied to its largest magnitude, so a block of
 *   G has the largest of the scales its groups of 32 would get on their own.  An
 *   all-zero block has scale -127, the bottom of the range (every integer satisfies
 *   the rule's inequality for a zero maximum), so it never raises a row's largest
 *   scale.
 */
#ifndef CURVEFP_H
#define CURVEFP_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    CURVEFP_E4C3 = 0,       /* 8 bits, E=4, C=3, 127 levels, H=8 */
    CURVEFP_E5C2 = 1,       /* 8 bits, E=5, C=2, 127 levels, H=4 */
    CURVEFP_E3C3 = 2,       /* 7 bits, E=3, C=3,  63 levels, H=8 */
    /* E4C3 with the rational radices of Tab. radix-frontier (Sec. 3.1: r = 2^{p/q},
     * levels r^{n/K} = 2^{p n/(qK)}, Eq. phase-count H = qK / gcd(p, qK)) */
    CURVEFP_E4C3_R8_9 = 3,  /* 8 bits, r = 2^{8/9}: levels 2^{n/9} in [2^-7, 2^7], H=9 */
    CURVEFP_E4C3_R3_4 = 4   /* 8 bits, r = 2^{3/4}: levels 2^{3n/32} in [2^-5.906, 2^5.906], H=32 */
} curvefp_format;

typedef enum {
    CURVEFP_F32 = 0,
    CURVEFP_BF16 = 1
} curvefp_dtype;

typedef enum {
    CURVEFP_OK = 0,
    CURVEFP_ERR_NULL = -1,     /* a required pointer is NULL */
    CURVEFP_ERR_SHAPE = -2,    /* non-positive or inconsistent sizes or counts, ld too small, blocked extent % block != 0 */
    CURVEFP_ERR_FORMAT = -3,   /* unknown format or dtype */
    CURVEFP_ERR_BLOCK = -4,    /* block not a positive multiple of 32, or block_axis not 0/1 */
    CURVEFP_ERR_ALIGN = -5,    /* pointer or row not 16-byte aligned */
    CURVEFP_ERR_HIP = -6       /* a kernel launch failed */
} curvefp_status;

/* Format parameters from Tab. curvefp-formats: element bits, E, C and the phase
 * count H = qK/gcd(p, qK) of Eq. phase-count (binary radix: H = K).  Any output
 * pointer may be NULL.  Returns CURVEFP_OK or CURVEFP_ERR_FORMAT. */
int curvefp_format_info(int format, int* bits, int* E, int* C, int* phases);

/* Radix r = 2^{p/q} of a format (p = q = 1: binary).  Returns CURVEFP_OK or
 * CURVEFP_ERR_FORMAT. */
int curvefp_format_radix(int format, int* p, int* q);

/* Bytes of the code array for `outer` rows of `k` elements each
 * (outer*k for E4C3/E5C2, outer*(k/32)*28 for E3C3); negative status on bad input. */
int64_t curvefp_codes_bytes(int format, int64_t outer, int64_t k, int block);

/* Number of int8 scales: outer * (k / block); negative status on bad input. */
int64_t curvefp_scales_count(int64_t outer, int64_t k, int block);

/*
 * Block quantization Q(X) (Sec. 3.1).
 *   src     [rows][ld_src] elements of `dtype` (fp32 or bf16), row-major.
 *   block_axis = 1: blocks of G run along each row; codes are [rows][cols]
 *                   (E3C3: [rows][cols/32][28] bytes), scales [rows][cols/G].
 *   block_axis = 0: blocks run down the columns (quantize-transpose); codes are
 *                   [cols][rows] (E3C3: [cols][rows/32][28]), scales [cols][rows/G].
 *   Blocks of 32..512 (a power of two) along rows are quantized in one pass; any
 *   other G, and every G > 32 down the columns, first write the block scales in
 *   a pass of their own (the source is read twice).
 * Scale (dynamic, ceil-absmax): a_b is the smallest integer with
 *   max|x| <= 2^{a_b} * fl32(2^{n_max/K}), clamped to [-127, 127]; -127 for an
 *   all-zero block; -128 (and all-zero codes) for a block holding NaN/Inf.
 * Element: the magnitude nearest to |x| 2^{-a_b} in absolute error among zero
 *   and the levels 2^{n/K}, saturating at the endpoints; the sign is kept,
 *   except that every zero result is the code 0.
 */
int curvefp_quantize(const void* src, int dtype, int64_t rows, int64_t cols, int64_t ld_src,
                     int block_axis, int format, int block,
                     void* codes, int8_t* scales, void* stream);

/*
 * Block quantization with static-operand scales (Sec. 3.1: a static operand takes the
 * power-of-two scale whose reconstruction has the least squared error), for weights quantized
 * once.  Same arguments, layouts and results as curvefp_quantize except the scale: each
 * block tries the scales a_c + u, a_c its ceil-absmax scale, for u = 0, -1, ...,
 * -(candidates - 1) and then, when the format's level pattern spans P > 1 octaves
 * (P = p / gcd(p, qK): 3 for CURVEFP_E4C3_R3_4, else 1), u = 1 .. P - 1 (a scale a_c + P + j
 * is never better than a_c + j); scales outside [-127, 127] are skipped.  Each candidate's
 * codes are reconstructed to fp32 exactly as curvefp_dequantize does, the squared errors
 * (x - x_hat)^2 are summed in fp64 over the block's 32 elements in index order, each
 * product and sum rounded once, and the first candidate in the order above with the least
 * sum wins.  candidates in [1, 8], else CURVEFP_ERR_SHAPE.  Any block size of curvefp_quantize
 * (the sums then run over the block's G elements in index order).  Zero blocks get scale -127 and
 * non-finite blocks -128 with zero codes, as in curvefp_quantize.
 */
int curvefp_quantize_mse(const void* src, int dtype, int64_t rows, int64_t cols, int64_t ld_src,
                         int block_axis, int format, int block, int candidates,
                         void* codes, int8_t* scales, void* stream);

/*
 * Tensorwise scale sharing (Sec. 3.1 evaluates tensorwise, rowwise and fixed-size blocks): one
 * ceil-absmax scale for the whole tensor, i.e. the block is the tensor.  Codes as
 * curvefp_quantize's for the same block_axis; the scale is written once per output row,
 * scales [outer] (outer = rows for block_axis = 1, cols for 0), all equal, so every consumer
 * takes the operand as rowwise-scaled (block = the blocked extent).  A NaN or infinity
 * anywhere poisons the tensor (scale -128, zero codes).
 *   workspace  one 32-bit word of device memory (4-byte aligned), scratch of the call:
 *              calls that share it must be ordered.
 * The blocked extent must be a multiple of 32 and at most 2^30 (CURVEFP_ERR_SHAPE).  The source
 * is read twice (its maximum, then the codes).
 */
int curvefp_quantize_tensorwise(const void* src, int dtype, int64_t rows, int64_t cols, int64_t ld_src,
                                int block_axis, int format, void* codes, int8_t* scales, void* workspace,
                                void* stream);

/*
 * Block quantization with S-bit scale exponents (Eq. effective-rate, R = 1 + E + C + S/G bits
 * per value; Sec. 4.2 prices E3C3 weights at S = 4 and activations at S = 5), blocks of G along
 * the rows of src.  The paper gives only the width; the layout taken here: each row keeps one
 * int8 reference e_r, the largest ceil-absmax scale among its blocks that are finite and not all
 * zero (0 if there is none), and each block an unsigned S-bit offset d = e_r - a', where
 * a' = max(a_b, e_r - (2^S - 2)) and a_b is the block's ceil-absmax scale: a block whose scale
 * lies more than 2^S - 2 below the reference is quantized at the raised scale a' (its smallest
 * values lose resolution, none saturates).  d = 2^S - 1 marks a block that held a NaN or an
 * infinity (its codes are zero); an all-zero block has d = 0.  Codes are curvefp_quantize's at
 * the scales a' (identical to curvefp_quantize's codes wherever no block is raised).
 *   codes    [rows][cols] bytes (E3C3: [rows][cols/32][28]), 16-byte aligned;
 *   row_ref  [rows] int8;
 *   offsets  [rows][curvefp_compact_offsets_bytes(1, cols, block, scale_bits)] bytes: offset j of
 *            a row at bits [S j, S j + S) of a little-endian bit string, rows padded to bytes.
 * scale_bits in [2, 8] and block a multiple of 32 (CURVEFP_ERR_BLOCK otherwise); cols % block
 * == 0 and cols <= 131072 (CURVEFP_ERR_SHAPE otherwise); src and rows 16-byte aligned.
 */
int64_t curvefp_compact_offsets_bytes(int64_t rows, int64_t cols, int block, int scale_bits);
int curvefp_quantize_compact(const void* src, int dtype, int64_t rows, int64_t cols, int64_t ld_src,
                             int format, int block, int scale_bits, void* codes, int8_t* row_ref,
                             uint8_t* offsets, void* stream);

/*
 * int8 block scales [rows][nblocks] from curvefp_quantize_compact's row references and packed
 * offsets: e_r - d, or -128 for the marker 2^S - 1.  With them, every entry point that takes
 * scales (dequantize, the GEMMs) consumes S-bit-scaled operands with block = G.
 */
int curvefp_scales_unpack(const int8_t* row_ref, const uint8_t* offsets, int64_t rows, int64_t nblocks,
                          int scale_bits, int8_t* scales, void* stream);

/*
 * Reconstruction x_hat = (-1)^s 2^{a_b} 2^{n/K} (Eq. curvefp-value), written as
 * the nearest fp32 value (ties to even).  codes/scales as produced by
 * curvefp_quantize with block_axis = 1 for an [outer][k] tensor;
 * dst [outer][ld_dst] fp32.  Zero codes give +0.0; poisoned blocks give NaN.
 */
int curvefp_dequantize(const void* codes, const int8_t* scales, int format,
                       int64_t outer, int64_t k, int block,
                       float* dst, int64_t ld_dst, void* stream);

/*
 * Size limits of the GEMM entry points (curvefp_gemm, curvefp_gemm_ws, the prepared calls,
 * curvefp_gemm_ws_static, curvefp_gemm_requant, curvefp_gemm_mixed and their byte counts):
 * K <= CURVEFP_MAX_K, and for curvefp_gemm also M <= CURVEFP_MAX_M_FUSED; larger sizes return
 * CURVEFP_ERR_SHAPE before anything is launched.  The expansion's grid has one workgroup row per
 * four K blocks of 32 and the fused kernel's one per 256 rows of A, at most 65535 each; within
 * these limits every kernel's byte offsets inside a tile of 256 rows stay below 2^31.
 */
#define CURVEFP_MAX_K ((int64_t)8388480)        /* 32 * 4 * 65535 */
#define CURVEFP_MAX_M_FUSED ((int64_t)16776960) /* 256 * 65535 */

/*
 * CurveFP GEMM: C[M][N] = deq(A)[M][K] . deq(B)[N][K]^T in fp32, the forward
 * contract Q_A(X) Q_W(W)^T of Sec. 3.3 with both operands K-contiguous
 * (A codes [M][K], B codes [N][K], scales [.][K/G], one format and one G for both).
 * c is [M][ldc] fp32, overwritten.
 *
 * Every nonzero product is, in the code domain, a sign xor, a curve-index sum
 * with carry into the exponent, an exponent sum and a scale sum
 * (Eq. curve-index-product); the dot product is the fixed-coefficient
 * reduction sum_h 2^{h/H} N_h of its phase sums (Eq. binned-accumulation).
 * The kernel evaluates that sum on the matrix cores: each code is expanded to
 * an fp16 high/low pair (22 significant bits) carrying its block scale
 * relative to the row's largest block scale, three f16 MFMA products
 * (hi.hi + hi.lo + lo.hi) accumulate in fp32, and the epilogue applies the
 * row and column scale offsets exactly.  Accumulation is fp32.  Relative
 * Frobenius error against the exact phase-binned sum is about 1e-7 on the
 * benchmark workloads.
 *
 * Non-finite sources: a block with scale -128 (it held a NaN or an infinity)
 * reconstructs to NaN, so, as deq(A) deq(B)^T in IEEE arithmetic (0 * NaN is
 * NaN), every output in a row of A or a column (row of B) that holds such a
 * block is NaN; the other outputs are unaffected.
 *
 * Scale-spread limit (the one place where the result can depart from the exact
 * sum by more than rounding).  Let alpha be the largest block scale of a row of
 * A (or of B) and top = 2^{alpha + e_max + 1}, e_max = floor(log2) of the
 * format's top level (7 for E4C3, 15 for E5C2, 3 for E3C3; all-zero blocks,
 * scale -127, and poisoned blocks never set alpha).  An element v of that row
 *   - with |v| >= 2^-18 top keeps 22 significant bits (each product is good
 *     to about 2^-21 relative);
 *   - with |v| < 2^-18 top keeps an absolute error of at most 2^-39 top;
 *   - with |v| < 2^-41 top is flushed: it contributes nothing.
 * A block loses all of its contribution only when its scale lies more than 41
 * binades below alpha; tests/test_gpu_accuracy_contract.py pins each clause.
 *
 * This entry point allocates nothing: the expansion happens inside the GEMM
 * kernel, once per workgroup that needs a code.  curvefp_gemm_ws below does the
 * expansion once per code and is faster; both give the same C bit for bit.
 */
int curvefp_gemm(const void* a_codes, const int8_t* a_scales,
                 const void* b_codes, const int8_t* b_scales,
                 int64_t M, int64_t N, int64_t K, int format, int block,
                 float* c, int64_t ldc, void* stream);

/*
 * Bytes of device workspace curvefp_gemm_ws needs for an M x N x K product
 * (4 bytes per element of A and B with rows padded to multiples of 256, plus
 * one int32 per padded row; when K is split in two -- fewer than 256 output
 * tiles of 256 x 256 and K >= 512 -- also 512 KiB of partial sums and one
 * arrival counter per tile).  Returns CURVEFP_ERR_SHAPE for non-positive
 * sizes or K not a multiple of 32.
 */
int64_t curvefp_gemm_workspace_bytes(int64_t M, int64_t N, int64_t K);

/*
 * The same product as curvefp_gemm (Sec. 3.3, Eq. binned-accumulation, same
 * arguments and result, bit for bit), through a caller-owned device workspace
 * of at least curvefp_gemm_workspace_bytes(M, N, K) bytes, 256-byte aligned.
 * The codes of A and B are first expanded once into fp16 high/low planes in
 * the workspace; the GEMM kernel then streams those planes into LDS and spends
 * its main loop on the matrix cores.  The workspace contents are scratch:
 * calls that share a workspace must be ordered (same stream, or synchronized).
 * Errors as curvefp_gemm, plus CURVEFP_ERR_NULL for a null workspace,
 * CURVEFP_ERR_SHAPE if workspace_bytes is too small and CURVEFP_ERR_ALIGN if
 * the workspace is not 256-byte aligned.
 */
int curvefp_gemm_ws(const void* a_codes, const int8_t* a_scales,
                    const void* b_codes, const int8_t* b_scales,
                    int64_t M, int64_t N, int64_t K, int format, int block,
                    float* c, int64_t ldc, void* workspace, int64_t workspace_bytes,
                    void* stream);

/*
 * Prepared operands: the staging step of curvefp_gemm_ws as a call of its own.  The GEMM
 * (Sec. 3.3, Eq. binned-accumulation) needs each operand's codes expanded into fp16 high/low
 * planes relative to its rows' largest block scales; that expansion depends on the operand
 * alone.  curvefp_prepare writes it for one operand into a caller-owned buffer, and
 * curvefp_gemm_prepared multiplies two prepared operands.  An operand that several products
 * share (static weights, Sec. 3.1) is then expanded once, and the two operands of one product
 * can be expanded on two streams, each as soon as it is quantized.
 * A backward GEMM's reused forward operand (Sec. 3.3: the codes kept from the forward pass, read
 * transposed) is prepared the same way with trans = 1.  prepare(A), prepare(B), gemm_prepared
 * give the C of curvefp_gemm_ws bit for bit, and for two formats or reused operands the C of
 * curvefp_gemm_mixed with the same trans_a and trans_b.
 *
 * curvefp_prepared_bytes: bytes of the prepared form of an operand with `rows` GEMM rows over
 * k (4 bytes per element with rows padded to a multiple of 256, plus one int32 per padded row;
 * trans = 1 adds 32 bytes per 256 rows per 256 k of scratch).  Returns CURVEFP_ERR_SHAPE for
 * non-positive sizes, k not a multiple of 32 or trans not 0 or 1.
 */
int64_t curvefp_prepared_bytes(int64_t rows, int64_t k, int trans);

/*
 * Expand one operand with `rows` GEMM rows over k, in `format`, into `prepared` (device,
 * 256-byte aligned, at least curvefp_prepared_bytes(rows, k, trans) bytes, passed in
 * prepared_size).  The codes and scales are those curvefp_quantize made
 *   trans = 0: of a [rows][k] tensor along k: codes [rows][k] (E3C3 [rows][k/32][28]), block
 *              scales [rows][k/block], k % block == 0;
 *   trans = 1: of a [k][rows] tensor along rows (a forward operand a backward GEMM reuses):
 *              codes [k][rows] (E3C3 [k][rows/32][28]), scales [k][rows/block],
 *              rows % block == 0 and rows <= 256 * 65535.  The buffer is overwritten with the expansion of the codes and
 * scales as they are when the call runs; it does not record its shape or format, so the GEMM
 * that reads it must be given the same rows (M or N), k and format.  Asynchronous on `stream`
 * (null: the null stream).
 * Errors: CURVEFP_ERR_NULL, _FORMAT, _BLOCK (block not a positive multiple of 32, trans not 0
 * or 1), _SHAPE (non-positive sizes, k % 32, the blocked extent not a multiple of block,
 * prepared_size too small), _ALIGN (codes not 16-byte or prepared not 256-byte aligned), _HIP
 * (a launch failed).
 */
int curvefp_prepare(const void* codes, const int8_t* scales, int64_t rows, int64_t k,
                    int format, int block, int trans, void* prepared, int64_t prepared_size,
                    void* stream);

/*
 * Quantize and prepare in one pass: Q(X) of Sec. 3.1 for a [rows][k] source with blocks along
 * k (curvefp_quantize with block_axis = 1), the result's prepared form for the GEMM (Sec. 3.3:
 * what curvefp_prepare writes from these codes with trans = 0) and, when dst is not null, its
 * reconstruction (Eq. curvefp-value: what curvefp_dequantize writes), from one read of the
 * source.  codes, scales, prepared and dst are bit for bit those of the three separate calls.
 *   src      [rows][ld_src] fp32 (dtype 0) or bf16 (dtype 1), 16-byte aligned rows.
 *   codes    [rows][k] (E3C3 [rows][k/32][28]), scales [rows][k/block], 16-byte aligned codes.
 *   prepared at least curvefp_prepared_bytes(rows, k, 0) bytes (prepared_size), 256-byte aligned.
 *   dst      null, or [rows][ld_dst] fp32 with 16-byte aligned rows.
 * Rows of up to 8192 bf16 or 4096 fp32 elements (bf16 rows of up to 16384 in tensors of at most
 * 2^26 elements), in tensors of fewer than 2^23 rows, take one launch: a wave or a workgroup
 * reads its row once, holds it in LDS while
 * it takes the block scales and the row's largest scale, then writes every output.  Other shapes
 * run the quantize, expansion and reconstruction kernels in turn (the same outputs; measured
 * faster there).  block is 32, 64, 128, 256 or 512 (other G: curvefp_quantize,
 * curvefp_prepare and curvefp_dequantize); k <= CURVEFP_MAX_K.  Errors:
 * CURVEFP_ERR_NULL (src, codes, scales or prepared), _FORMAT (dtype or format), _BLOCK, _SHAPE
 * (non-positive sizes, k % block, k > CURVEFP_MAX_K, ld_src < k, ld_dst < k, prepared_size too
 * small, rows >= 2^31), _ALIGN, _HIP.
 */
int curvefp_quantize_prepare(const void* src, int dtype, int64_t rows, int64_t k, int64_t ld_src,
                             int format, int block, void* codes, int8_t* scales,
                             void* prepared, int64_t prepared_size, float* dst, int64_t ld_dst,
                             void* stream);

/*
 * curvefp_quantize_prepare of the two operands of one GEMM in one launch (Sec. 3.3: both operands
 * of Q_A(X) Q_W(W)^T are quantized along the contraction axis k; one format, one block size and
 * one source type for both): A [rows_a][ld_a] and B [rows_b][ld_b], each with its own codes,
 * scales, prepared buffer (prepared_a_size / prepared_b_size bytes) and optional reconstruction
 * (dst_a / dst_b, null for none).  The outputs are those of two curvefp_quantize_prepare calls,
 * bit for bit; one launch spreads both operands over the whole GPU and needs no second stream.
 * When the two together fall outside the one-launch shapes above (rows_a + rows_b rows over k),
 * each operand runs as curvefp_quantize_prepare would run it, A then B, on the same stream.
 * Errors: those of curvefp_quantize_prepare for either operand, and CURVEFP_ERR_SHAPE for
 * rows_a + rows_b >= 2^31.
 */
int curvefp_quantize_prepare_pair(const void* src_a, int64_t rows_a, int64_t ld_a, void* codes_a,
                                  int8_t* scales_a, void* prepared_a, int64_t prepared_a_size,
                                  float* dst_a, int64_t ld_dst_a,
                                  const void* src_b, int64_t rows_b, int64_t ld_b, void* codes_b,
                                  int8_t* scales_b, void* prepared_b, int64_t prepared_b_size,
                                  float* dst_b, int64_t ld_dst_b,
                                  int dtype, int64_t k, int format, int block, void* stream);

/*
 * Bytes of device workspace curvefp_gemm_prepared needs for an M x N x K product: 0 unless K
 * is split in two (fewer than 256 output tiles of 256 x 256 and K >= 512; then one arrival
 * counter per tile and 512 KiB of partial sums per tile).  CURVEFP_ERR_SHAPE for non-positive
 * sizes or K not a multiple of 32.
 */
int64_t curvefp_gemm_prepared_workspace_bytes(int64_t M, int64_t N, int64_t K);

/*
 * C[M][N] = deq(A) deq(B)^T in fp32 (the contract of curvefp_gemm, including its non-finite
 * and scale-spread clauses) from A prepared with M rows over K in format_a and B prepared with
 * N rows over K in format_b (each by curvefp_prepare, either trans; the formats may differ).
 * c is [M][ldc] fp32, overwritten.  workspace: at least
 * curvefp_gemm_prepared_workspace_bytes(M, N, K) bytes, 256-byte aligned (may be null when
 * that is 0); its contents are scratch, so calls that share it must be ordered.  The prepared buffers are only read: one prepared operand may serve
 * concurrent calls.  Errors: CURVEFP_ERR_NULL, _FORMAT, _SHAPE (non-positive sizes, K % 32,
 * ldc < N, workspace too small), _ALIGN (prepared buffers or workspace not 256-byte aligned,
 * c not 16-byte aligned), _HIP.
 */
int curvefp_gemm_prepared(const void* a_prepared, int format_a,
                          const void* b_prepared, int format_b,
                          int64_t M, int64_t N, int64_t K, float* c, int64_t ldc,
                          void* workspace, int64_t workspace_bytes, void* stream);

/* Bytes of the device scratch curvefp_gemm_ws_static uses on each GPU. */
#define CURVEFP_STATIC_SCRATCH_BYTES ((int64_t)128 << 20)

/*
 * For callers that cannot allocate device memory (code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc): curvefp_gemm_ws with the library's own static
 * device scratch as its workspace.  Same operands, result (bit for bit) and errors as
 * curvefp_gemm_ws, without the workspace arguments.  The scratch is one 256-byte aligned array
 * of CURVEFP_STATIC_SCRATCH_BYTES per GPU, part of the library's code object: each GPU the
 * entry point runs on holds it from the first call on that device until the process ends.
 * The call makes no hipMalloc, hipFree or other allocation; its first call on a device looks
 * up the array's device address (hipGetSymbolAddress) and keeps it.
 *   Limit: curvefp_gemm_workspace_bytes(M, N, K) <= CURVEFP_STATIC_SCRATCH_BYTES, else
 *   CURVEFP_ERR_SHAPE (before any HIP call).
 *   Every call on one GPU uses that GPU's array, and everything the kernels need cleared is
 *   cleared by the call itself; calls that overlap on one GPU (different streams, or host
 *   threads without ordering) race on the array and may return wrong results.
 */
int curvefp_gemm_ws_static(const void* a_codes, const int8_t* a_scales,
                           const void* b_codes, const int8_t* b_scales,
                           int64_t M, int64_t N, int64_t K, int format, int block,
                           float* c, int64_t ldc, void* stream);

/*
 * The product of curvefp_gemm_ws (same operands, format, workspace and fp32 values), with
 * the output requantized in the GEMM's epilogue instead of stored as fp32: the explicit
 * output requantization of Sec. 3.2 (products are closed on widened coordinates; only the
 * requantization to a finite destination may saturate).  C is quantized in blocks of
 * out_block consecutive outputs along each row into out_format with the rule of
 * curvefp_quantize (ceil-absmax scale, nearest level), so out_codes / out_scales equal
 * curvefp_quantize (block_axis = 1, block = out_block) of the fp32 C that curvefp_gemm_ws
 * returns, bit for bit.
 *   out_codes [M][N] bytes (E3C3: [M][N/32][28]), out_scales [M][N/out_block].
 * out_block is 32, 64, 128 or 256 (an output block lies within one 256-column tile of the
 * epilogue; CURVEFP_ERR_BLOCK otherwise); N must be a multiple of out_block
 * (CURVEFP_ERR_SHAPE otherwise); out_codes 16-byte aligned.  Other errors as curvefp_gemm_ws.
 */
int curvefp_gemm_requant(const void* a_codes, const int8_t* a_scales,
                         const void* b_codes, const int8_t* b_scales,
                         int64_t M, int64_t N, int64_t K, int format, int block, int out_format,
                         int out_block, void* out_codes, int8_t* out_scales,
                         void* workspace, int64_t workspace_bytes, void* stream);

/*
 * Bytes of device workspace curvefp_gemm_mixed needs for an M x N x K product:
 * curvefp_gemm_workspace_bytes(M, N, K) plus, per operand, 4 bytes per
 * (256-row slab of K, 32 padded GEMM rows) for the column maxima of a reused
 * operand's scales.  CURVEFP_ERR_SHAPE for non-positive sizes or K % 32 != 0.
 */
int64_t curvefp_gemm_mixed_workspace_bytes(int64_t M, int64_t N, int64_t K);

/*
 * CurveFP GEMM of two operands that may differ in format and in how their
 * codes are stored: the backward GEMMs of Sec. 3.3, which multiply E5C2 output
 * gradients Q_G(dY) with the E4C3 codes kept from the forward pass,
 *   dX = Q_G(dY) Q_W(W)      (A = dY codes, B = the forward W codes, b_trans = 1)
 *   dW = Q_G(dY)^T Q_A(X)    (A = dY codes, a_trans = 1; B = the forward X codes, b_trans = 1).
 *   C[M][N] = deq(A)[M][K] . deq(B)[N][K]^T in fp32, c [M][ldc], overwritten.
 * Operand layouts (per operand, X = A with R = M or X = B with R = N):
 *   x_trans = 0: the codes and scales curvefp_quantize(block_axis = 1) makes of an
 *                [R][K] tensor: codes [R][K] (E3C3 [R][K/32][28]), scales [R][K/G];
 *   x_trans = 1: those it makes of a [K][R] tensor: codes [K][R] (E3C3 [K][R/32][28]),
 *                scales [K][R/G]; the blocks lie along R, so R % G == 0.
 *   Both operands use the same block size G; K % 32 == 0, and K % G == 0 when an
 *   operand is quantized along K.
 * Formats a_format, b_format are any of the three.  The product of two curve
 * values with curve counts K_a, K_b (both powers of two) is a value of the finer
 * lattice L = max(K_a, K_b): indices lift as n' = (L / K) n, the phase is
 * h = (n'_a + n'_b) mod L and the carry joins the exponent (Eq. curve-index-product
 * with one lattice for both); the sum is sum_h 2^{h/L} N_h.  Evaluated on the matrix
 * cores as in curvefp_gemm_ws: every element is expanded once to an fp16 high/low
 * pair carrying its own scale relative to its row's largest, with the error bound
 * stated for curvefp_gemm.  With a_trans = b_trans = 0 and a_format == b_format the
 * result equals curvefp_gemm_ws's bit for bit.  A GEMM row (of A or B) any of whose
 * elements lies in a block with scale -128 gives NaN outputs, as in curvefp_gemm.
 * Errors: as curvefp_gemm_ws, plus CURVEFP_ERR_BLOCK for a trans flag other than
 * 0/1 and CURVEFP_ERR_SHAPE for a reused operand with R % G != 0, more than
 * 65535 256-row tiles of reused operands, or a workspace smaller than
 * curvefp_gemm_mixed_workspace_bytes(M, N, K).  The workspace (256-byte aligned)
 * is scratch: calls that share it must be ordered.
 */
int curvefp_gemm_mixed(const void* a_codes, const int8_t* a_scales, int a_format, int a_trans,
                       const void* b_codes, const int8_t* b_scales, int b_format, int b_trans,
                       int64_t M, int64_t N, int64_t K, int block, float* c, int64_t ldc,
                       void* workspace, int64_t workspace_bytes, void* stream);

/* Static description of a status code. */
const char* curvefp_status_string(int status);

#ifdef __cplusplus
}
#endif

#endif /* CURVEFP_H */
