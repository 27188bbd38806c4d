/*
 * curvefp_oracle.c -- exact CurveFP GEMM on the CPU.
 *
 * TEST INFRASTRUCTURE ONLY: loaded by the oracle package for tests, smoke()
 * and the cpu_baseline leg of bench.py.  It shares no code with the HIP library.
 *
 * For every output C[i][j] = sum_k x_hat(A[i][k]) * x_hat(B[j][k]) the
 * products are formed in the code domain and accumulated exactly in signed
 * integer bins, as the paper's constructive realization describes
 * (Sec. 3.2 "Constructive arithmetic realization", App. A.1):
 *
 *   u     = p (n_x + n_w)
 *   delta = (-1)^(s_x xor s_w)
 *   h     = (u mod qK) / g,            g = gcd(p, qK)
 *   t     = a_x + a_w + floor(u / qK)
 *   A[h][t] += delta                   (a zero operand suppresses the update)
 *
 * and the dot product is sum_h 2^(h/H) sum_t A[h][t] 2^t (Eq. binned-accumulation).
 * The per-phase sums N_h = sum_t A[h][t] 2^t are formed exactly as two's
 * complement big integers; only the last step, sum_h 2^(h/H) N_h with the
 * irrational phase weights, is rounded, in __float128 (113-bit significand).
 *
 * Codes are unpacked (one per byte): code = s << (E+C) | m, m = n + B, m = 0 is
 * zero.  Scales are int8 power-of-two exponents, one per `block` consecutive
 * elements along k.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <quadmath.h>
#include <omp.h>

typedef struct {
    int E, C, p, q;
    int K, B, QK, g, H, mag_mask;
} fmt_t;

static int gcd_i(int a, int b) {
    while (b) { int r = a % b; a = b; b = r; }
    return a < 0 ? -a : a;
}

static int floor_div(int a, int b) { int d = a / b; if ((a % b != 0) && ((a < 0) != (b < 0))) d--; return d; }
static int floor_mod(int a, int b) { return a - b * floor_div(a, b); }

static int make_fmt(int E, int C, int p, int q, fmt_t* f) {
    if (E < 1 || C < 0 || E + C > 7 || p < 1 || q < 1) return -1;
    f->E = E; f->C = C; f->p = p; f->q = q;
    f->K = 1 << C;
    f->B = 1 << (E + C - 1);
    f->QK = q * f->K;
    f->g = gcd_i(p, f->QK);
    f->H = f->QK / f->g;
    f->mag_mask = (1 << (E + C)) - 1;
    return 0;
}

/* ---- exact signed big integers: little-endian uint32 limbs, two's complement ---- */
#define NLIMB 24 /* 768 bits: holds sum_t A[h][t] 2^(t - t_lo) for any t span we can meet */

static void big_add_shifted(uint32_t* x, int64_t v, int shift) {
    /* x += v * 2^shift, v signed with |v| < 2^31 */
    int j = shift / 32, off = shift % 32;
    int64_t w = v * ((int64_t)1 << off);          /* |w| < 2^63 */
    uint64_t carry = 0;
    uint32_t ext = (w < 0) ? 0xFFFFFFFFu : 0u;
    uint32_t add0 = (uint32_t)((uint64_t)w & 0xFFFFFFFFu);
    uint32_t add1 = (uint32_t)(((uint64_t)w >> 32) & 0xFFFFFFFFu);
    for (int l = j; l < NLIMB; l++) {
        uint32_t a = (l == j) ? add0 : (l == j + 1) ? add1 : ext;
        uint64_t s = (uint64_t)x[l] + a + carry;
        x[l] = (uint32_t)s;
        carry = s >> 32;
    }
}

/* Two's complement big integer -> __float128, rounded to odd at 113 bits, so that
 * a later rounding to float64 (53 bits) is the correct rounding of the integer. */
static __float128 big_to_f128(const uint32_t* x) {
    uint32_t y[NLIMB];
    int neg = (x[NLIMB - 1] >> 31) & 1;
    memcpy(y, x, sizeof(y));
    if (neg) { /* y = -x */
        uint64_t carry = 1;
        for (int l = 0; l < NLIMB; l++) {
            uint64_t s = (uint64_t)(uint32_t)(~y[l]) + carry;
            y[l] = (uint32_t)s;
            carry = s >> 32;
        }
    }
    int top = NLIMB - 1;
    while (top >= 0 && y[top] == 0) top--;
    if (top < 0) return 0;
    /* gather the four limbs from the top into a 128-bit window; lower limbs -> sticky */
    unsigned __int128 w = 0;
    int sticky = 0;
    for (int l = top; l > top - 4; l--) w = (w << 32) | (l >= 0 ? y[l] : 0u);
    for (int l = top - 4; l >= 0; l--) sticky |= (y[l] != 0);
    int lsb_exp = (top - 3) * 32;              /* weight of bit 0 of w */
    int bl = 0;
    for (unsigned __int128 t = w; t; t >>= 1) bl++;
    if (bl > 113) {
        int sh = bl - 113;
        unsigned __int128 dropped = w & ((((unsigned __int128)1) << sh) - 1);
        sticky |= (dropped != 0);
        w >>= sh;
        lsb_exp += sh;
    }
    if (sticky) w |= 1;                        /* round to odd */
    __float128 v = ldexpq((__float128)w, lsb_exp);
    return neg ? -v : v;
}

/* ---- per-output histogram of the bins A[h][t] ---- */
typedef struct {
    int H, t_min, t_span;
    int32_t* cnt;     /* [H][t_span] */
    int lo, hi;       /* touched range of t (relative), for clearing */
} hist_t;

static void hist_init(hist_t* hs, const fmt_t* f) {
    /* t = a_x + a_w + floor(u / qK), a in [-128, 127], |u| <= 2 p (B - 1) */
    int umax = 2 * f->p * (f->B - 1);
    int fmin = floor_div(-umax, f->QK), fmax = floor_div(umax, f->QK);
    hs->H = f->H;
    hs->t_min = -256 + fmin;
    hs->t_span = (254 + fmax) - hs->t_min + 1;
    hs->cnt = (int32_t*)calloc((size_t)f->H * hs->t_span, sizeof(int32_t));
    hs->lo = hs->t_span; hs->hi = -1;
}

static void hist_clear(hist_t* hs) {
    if (hs->hi >= hs->lo)
        for (int h = 0; h < hs->H; h++)
            memset(hs->cnt + (size_t)h * hs->t_span + hs->lo, 0, sizeof(int32_t) * (hs->hi - hs->lo + 1));
    hs->lo = hs->t_span; hs->hi = -1;
}

/* accumulate one dot product of length kd into the bins; returns max |A[h][t]| */
static void dot_bins(const fmt_t* f, hist_t* hs,
                     const uint8_t* a, const int8_t* as, const uint8_t* b, const int8_t* bs,
                     int64_t kd, int block) {
    const int EC = f->E + f->C;
    for (int64_t k = 0; k < kd; k++) {
        int ma = a[k] & f->mag_mask, mb = b[k] & f->mag_mask;
        if (ma == 0 || mb == 0) continue;                 /* zero sentinel: no update */
        int sx = (a[k] >> EC) & 1, sw = (b[k] >> EC) & 1;
        int nx = ma - f->B, nw = mb - f->B;
        int u = f->p * (nx + nw);
        int h = floor_mod(u, f->QK) / f->g;
        int t = as[k / block] + bs[k / block] + floor_div(u, f->QK);
        int rel = t - hs->t_min;
        hs->cnt[(size_t)h * hs->t_span + rel] += (sx ^ sw) ? -1 : 1;
        if (rel < hs->lo) hs->lo = rel;
        if (rel > hs->hi) hs->hi = rel;
    }
}

/* N_h = sum_t A[h][t] 2^t exactly, then V = sum_h 2^(h/H) N_h */
static __float128 reduce_bins(const fmt_t* f, const hist_t* hs, int32_t* max_count, __float128* phase_out) {
    __float128 v = 0;
    for (int h = 0; h < f->H; h++) {
        uint32_t big[NLIMB];
        memset(big, 0, sizeof(big));
        const int32_t* row = hs->cnt + (size_t)h * hs->t_span;
        for (int rel = hs->lo; rel <= hs->hi; rel++) {
            int32_t c = row[rel];
            if (!c) continue;
            if (max_count) { int32_t ac = c < 0 ? -c : c; if (ac > *max_count) *max_count = ac; }
            big_add_shifted(big, c, rel - hs->lo);
        }
        __float128 nh = ldexpq(big_to_f128(big), hs->lo + hs->t_min);
        if (phase_out) phase_out[h] = nh;
        v += exp2q((__float128)h / (__float128)f->H) * nh;
    }
    return v;
}

/*
 * C[i][j] (float64) for i in [0, M), j in [0, N).
 * a_codes [M][kd], a_scales [M][kd/block], b_codes [N][kd], b_scales [N][kd/block].
 * Returns 0, or -1 on bad arguments.  max_count (optional) receives max |A[h][t]|.
 */
int oracle_gemm_exact(const uint8_t* a_codes, const int8_t* a_scales,
                      const uint8_t* b_codes, const int8_t* b_scales,
                      int64_t M, int64_t N, int64_t kd, int block,
                      int E, int C, int p, int q,
                      double* out, int nthreads, int32_t* max_count) {
    fmt_t f;
    if (make_fmt(E, C, p, q, &f) || M < 0 || N < 0 || kd < 0 || block <= 0 || kd % block) return -1;
    if (nthreads > 0) omp_set_num_threads(nthreads);
    int32_t gmax = 0;
    #pragma omp parallel
    {
        hist_t hs;
        hist_init(&hs, &f);
        int32_t lmax = 0;
        #pragma omp for schedule(dynamic, 1)
        for (int64_t i = 0; i < M; i++) {
            for (int64_t j = 0; j < N; j++) {
                dot_bins(&f, &hs, a_codes + i * kd, a_scales + i * (kd / block),
                         b_codes + j * kd, b_scales + j * (kd / block), kd, block);
                __float128 v = reduce_bins(&f, &hs, &lmax, NULL);
                out[i * N + j] = (double)v;
                hist_clear(&hs);
            }
        }
        #pragma omp critical
        { if (lmax > gmax) gmax = lmax; }
        free(hs.cnt);
    }
    if (max_count) *max_count = gmax;
    return 0;
}

/* Phase sums N_h (as float64) of one dot product, for the phase-schedule tests. */
int oracle_dot_phase_sums(const uint8_t* a, const int8_t* as, const uint8_t* b, const int8_t* bs,
                          int64_t kd, int block, int E, int C, int p, int q,
                          double* phase_sums /* [H] */, double* value, int32_t* max_count) {
    fmt_t f;
    if (make_fmt(E, C, p, q, &f) || kd < 0 || block <= 0 || kd % block) return -1;
    hist_t hs;
    hist_init(&hs, &f);
    dot_bins(&f, &hs, a, as, b, bs, kd, block);
    __float128 ph[64];
    int32_t mc = 0;
    __float128 v = reduce_bins(&f, &hs, &mc, ph);
    for (int h = 0; h < f.H && h < 64; h++) phase_sums[h] = (double)ph[h];
    if (value) *value = (double)v;
    if (max_count) *max_count = mc;
    free(hs.cnt);
    return 0;
}

/*
 * Mixed-format GEMM (the backward recipe of Sec. 3.3: E5C2 output gradients times reused
 * E4C3 forward operands).  The paper states the closed product for one lattice.  Operand x has
 * magnitudes 2^(p_x n_x / N_x), N_x = q_x K_x; over the common denominator D = lcm(N_a, N_b)
 * both exponents are integers over D: u_x = p_x (D / N_x) n_x, and the product's exponent is
 * (u_a + u_b) / D, so its address is
 *   u = u_a + u_b,  h = (u mod D) / g,  t = a_a + a_b + floor(u / D),  delta = (-1)^(s_a xor s_b),
 * with g = gcd(p_a D / N_a, p_b D / N_b, D) and H = D / g phases: the single-format rule when
 * the formats agree.  For binary radices (N = K, powers of two) D = max(K_a, K_b) and the lift
 * is n' = (D / K) n.  Scales are per element here (a_scales [M][kd], b_scales [N][kd]): callers
 * whose blocks lie along k expand them, and operands whose blocks lie along the other axis
 * (forward codes reused in a backward GEMM) are passed the same way.
 */
typedef struct {
    int D, g, H, la, lb;   /* common denominator, phase divisor, phases, exponent multipliers */
} lattice_t;

static void dot_bins_mixed(const fmt_t* fx, const fmt_t* fw, const lattice_t* L, hist_t* hs,
                           const uint8_t* a, const int8_t* as, const uint8_t* b, const int8_t* bs, int64_t kd) {
    const int ECx = fx->E + fx->C, ECw = fw->E + fw->C;
    for (int64_t k = 0; k < kd; k++) {
        int ma = a[k] & fx->mag_mask, mb = b[k] & fw->mag_mask;
        if (ma == 0 || mb == 0) continue;
        int sx = (a[k] >> ECx) & 1, sw = (b[k] >> ECw) & 1;
        int u = L->la * (ma - fx->B) + L->lb * (mb - fw->B);
        int h = floor_mod(u, L->D) / L->g;
        int t = as[k] + bs[k] + floor_div(u, L->D);
        int rel = t - hs->t_min;
        hs->cnt[(size_t)h * hs->t_span + rel] += (sx ^ sw) ? -1 : 1;
        if (rel < hs->lo) hs->lo = rel;
        if (rel > hs->hi) hs->hi = rel;
    }
}

int oracle_gemm_exact_mixed(const uint8_t* a_codes, const int8_t* a_scales, int Ea, int Ca, int pa, int qa,
                            const uint8_t* b_codes, const int8_t* b_scales, int Eb, int Cb, int pb, int qb,
                            int64_t M, int64_t N, int64_t kd, double* out, int nthreads, int32_t* max_count) {
    fmt_t fx, fw, fl;
    if (make_fmt(Ea, Ca, pa, qa, &fx) || make_fmt(Eb, Cb, pb, qb, &fw) || M < 0 || N < 0 || kd < 0) return -1;
    lattice_t L;
    L.D = fx.QK / gcd_i(fx.QK, fw.QK) * fw.QK;
    L.la = pa * (L.D / fx.QK);
    L.lb = pb * (L.D / fw.QK);
    L.g = gcd_i(gcd_i(L.la, L.lb), L.D);
    L.H = L.D / L.g;
    if (L.H > 64 * 8) return -1;
    /* bins sized for the common lattice: |u| <= la (B_a - 1) + lb (B_b - 1), phases H over D */
    fl.E = 0; fl.C = 0; fl.p = 1; fl.q = 1; fl.K = L.D; fl.QK = L.D; fl.g = L.g; fl.H = L.H; fl.mag_mask = 0;
    fl.B = (L.la * (fx.B - 1) + L.lb * (fw.B - 1) + 1) / 2 + 1;
    if (nthreads > 0) omp_set_num_threads(nthreads);
    int32_t gmax = 0;
    #pragma omp parallel
    {
        hist_t hs;
        hist_init(&hs, &fl);
        int32_t lmax = 0;
        #pragma omp for schedule(dynamic, 1)
        for (int64_t i = 0; i < M; i++) {
            for (int64_t j = 0; j < N; j++) {
                dot_bins_mixed(&fx, &fw, &L, &hs, a_codes + i * kd, a_scales + i * kd,
                               b_codes + j * kd, b_scales + j * kd, kd);
                __float128 v = reduce_bins(&fl, &hs, &lmax, NULL);
                out[i * N + j] = (double)v;
                hist_clear(&hs);
            }
        }
        #pragma omp critical
        { if (lmax > gmax) gmax = lmax; }
        free(hs.cnt);
    }
    if (max_count) *max_count = gmax;
    return 0;
}

int oracle_max_threads(void) { return omp_get_max_threads(); }
