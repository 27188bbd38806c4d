// Host construction of libcurvefp's constant tables (run at build time by gen_tables.cpp).
//
// All irrational constants 2^{r/N} come from x87 80-bit exp2l (64-bit
// significand).  Every integer decision taken from them (a threshold floor, a
// rounding direction) is checked to sit far from the ambiguous point, so the
// 64-bit approximation cannot flip it; a failed check makes build_tables
// return false and the library refuses to run.
//
// Levels (Eq. curvefp-value with r = 2^{p/q}): a magnitude rank m = n + B
// stands for 2^{p n / N}, N = qK, i.e. 2^{w + f/N} with w = floor(p n / N) and
// f = p n mod N; binary radix is p = q = 1 (2^{e + k/K}).
//
// Quantizer (Sec. 3.1): the magnitude y is nearest to level n + 1 rather than n
// exactly when y exceeds the midpoint (2^{p n/N} + 2^{p (n+1)/N}) / 2, and to the
// smallest level rather than zero when y reaches half of it.  Each decision point
// is held as (octave o, 24-bit significand threshold T): y = M 2^{o-23} is above
// it iff (o_y, M) > (o, T).  The midpoints between levels are irrational (sums of
// distinct powers 2^{j/N}, linearly independent over Q), so no M sits on one; the
// zero point is irrational too, except when the smallest level is a power of two
// (r = 2^{8/9}: 2^{-7}), where it is the float 2^{w-1} and a tie goes to the level.
#include <cmath>
#include <cstdio>
#include <cstring>

#include "tables.hpp"

namespace curvefp {
namespace {

long double pow2frac(int f, int N) { return exp2l((long double)f / (long double)N); }

// floor(x) where x is known to lie far from an integer
bool safe_floor(long double x, int64_t* out) {
    long double f = floorl(x);
    long double fr = x - f;
    if (fr < 1e-7L || fr > 1.0L - 1e-7L) return false;
    *out = (int64_t)f;
    return true;
}

int floor_div(int a, int b) { return a / b - ((a % b != 0) && ((a < 0) != (b < 0)) ? 1 : 0); }

struct Point {
    int o;          // octave: the point lies in [2^o, 2^{o+1})
    int64_t T;      // significand threshold in [2^23, 2^24)
    bool exact;     // the point is the float T 2^{o-23} itself (ties go up)
};

struct Rule {
    int P, N, B, nmin, nmax;
    int nmid;
    Point mid[256];   // mid[n - nmin]: between levels n and n + 1
    Point zero;       // half the smallest level
};

// the irrational point v (> 0) as (octave, floor of its significand)
bool inexact_point(long double v, Point* pt) {
    int e2;
    frexpl(v, &e2);                 // v = f 2^e2, f in [0.5, 1)
    pt->o = e2 - 1;
    pt->exact = false;
    return safe_floor(ldexpl(v, 23 - pt->o), &pt->T);
}

long double level(const Rule& r, int n) {
    const int u = r.P * n;
    const int w = floor_div(u, r.N);
    return ldexpl(pow2frac(u - w * r.N, r.N), w);
}

bool make_rule(int E, int C, int P, int Q, Rule* r) {
    const int K = 1 << C;
    r->P = P;
    r->N = Q * K;
    r->B = 1 << (E + C - 1);
    r->nmin = -(r->B - 1);
    r->nmax = r->B - 1;
    r->nmid = r->nmax - r->nmin;
    if (r->nmid > 256) return false;
    for (int n = r->nmin; n < r->nmax; n++)
        if (!inexact_point(0.5L * (level(*r, n) + level(*r, n + 1)), &r->mid[n - r->nmin])) return false;
    const int u = P * r->nmin;
    const int w = floor_div(u, r->N);
    if (u - w * r->N == 0) {
        r->zero.o = w - 1;
        r->zero.T = (int64_t)1 << 23;
        r->zero.exact = true;
    } else if (!inexact_point(0.5L * level(*r, r->nmin), &r->zero)) {
        return false;
    }
    return true;
}

bool above(int o, int64_t M, const Point& p) {
    return o > p.o || (o == p.o && (p.exact ? M >= p.T : M > p.T));
}

// magnitude rank (0 = zero) of y = M 2^{o - 23}
int rank_of(const Rule& r, int o, int64_t M) {
    if (!above(o, M, r.zero)) return 0;
    int c = 0;
    for (int i = 0; i < r.nmid; i++) c += above(o, M, r.mid[i]) ? 1 : 0;
    return r.nmin + c + r.B;
}

// nearest fp16 (ties to even) of v >= 0; returns bits
bool rn_fp16(long double v, uint16_t* bits) {
    if (v == 0) { *bits = 0; return true; }
    int e2;
    frexpl(v, &e2);             // v = f 2^e2, f in [0.5, 1)
    int ex = e2 - 1;            // v in [2^ex, 2^{ex+1})
    int shift = (ex >= -14) ? (10 - ex) : 24;   // units of the last kept bit
    long double q = ldexpl(v, shift);
    long double fl = floorl(q);
    long double fr = q - fl;
    if (fabsl(fr - 0.5L) < 1e-9L && fr != 0.5L) return false;
    uint32_t qi = (uint32_t)fl;
    if (fr > 0.5L || (fr == 0.5L && (qi & 1))) qi++;
    if (ex >= -14) {
        if (qi == 2048) { qi = 1024; ex++; }
        if (ex + 15 >= 31) return false;
        *bits = (uint16_t)(((ex + 15) << 10) | (qi - 1024));
    } else {
        *bits = (uint16_t)qi;   // subnormal, or the smallest normal when qi == 1024
    }
    return true;
}

long double fp16_value(uint16_t b) {
    int e = (b >> 10) & 31, m = b & 1023;
    long double v = (e == 0) ? ldexpl((long double)m, -24) : ldexpl((long double)(1024 + m), e - 25);
    return (b & 0x8000) ? -v : v;
}

// mantissa field of fl32(2^{f/N}) and floor(2^{f/N} 2^62), with the checks that make both exact
bool significands(int f, int N, uint32_t* mant, uint64_t* sig62) {
    long double s = pow2frac(f, N);
    long double q = ldexpl(s, 23);
    long double fl = floorl(q), fr = q - fl;
    if (f && fabsl(fr - 0.5L) < 1e-9L) return false;
    uint32_t qi = (uint32_t)fl + (fr > 0.5L ? 1u : 0u);
    if (qi >= (1u << 24)) return false;
    *mant = qi - (1u << 23);
    *sig62 = (uint64_t)floorl(ldexpl(s, 62));
    // the subnormal reconstruction rounds sig62 at bit positions 40..63
    for (int sh = 40; sh <= 63 && f; sh++) {
        uint64_t rem = *sig62 & ((1ull << sh) - 1);
        uint64_t half = 1ull << (sh - 1);
        uint64_t d = rem > half ? rem - half : half - rem;
        if (d < 4) return false;
    }
    return true;
}

bool build_format(int E, int C, int P, int Q, FormatTables* ft) {
    Rule r;
    if (!make_rule(E, C, P, Q, &r)) return false;
    const int K = 1 << C, N = r.N;
    const int EC = E + C;
    ft->K = K;
    ft->P = P;
    ft->Q = Q;
    const int ohi = floor_div(P * r.nmax, N);           // octave of the top level
    const int oz = r.zero.o;                             // octave of the zero point
    ft->qlut_size = (ohi - oz + 1) * 128;
    if (ft->qlut_size > QLUT_MAX) return false;
    for (int i = 0; i < ft->qlut_size; i++) {
        int o = oz + i / 128;
        int64_t M0 = (int64_t)(128 + i % 128) << 16;
        int c0 = rank_of(r, o, M0), c1 = rank_of(r, o, M0 + 0xFFFF);
        uint32_t thr = 0xFFFF;
        if (c1 != c0) {
            if (c1 != c0 + 1) return false;  // at most one decision point per bucket
            int lo = 0, hi = 0xFFFF;          // largest low part that keeps c0
            while (lo < hi) {
                int mid = (lo + hi + 1) / 2;
                if (rank_of(r, o, M0 + mid) == c0) lo = mid; else hi = mid - 1;
            }
            thr = (uint32_t)lo;
        }
        ft->qlut[i] = ((uint32_t)c0 << 16) | thr;
    }
    for (int i = ft->qlut_size; i < QLUT_MAX; i++) ft->qlut[i] = 0;
    // binary radix: fl32(2^{k/K}) mantissas and 62-bit significands indexed by k
    for (int k = 0; k < 8; k++) { ft->mant[k] = 0; ft->sig62[k] = 0; }
    if (P == 1 && Q == 1)
        for (int k = 0; k < K; k++)
            if (!significands(k, K, &ft->mant[k], &ft->sig62[k])) return false;
    // every format: per magnitude rank, (w << 24) | mantissa of fl32(2^{f/N}) and the 62-bit
    // significand, for 2^{p n / N} = 2^{w + f/N}
    memset(ft->dq_em, 0, sizeof(ft->dq_em));
    memset(ft->dq_sig62, 0, sizeof(ft->dq_sig62));
    for (int m = 1; m < (1 << EC); m++) {
        const int u = P * (m - r.B);
        const int w = floor_div(u, N), f = u - w * N;
        uint32_t mant;
        uint64_t s62;
        if (!significands(f, N, &mant, &s62)) return false;
        ft->dq_em[m] = ((uint32_t)(w & 0xFF) << 24) | mant;
        ft->dq_sig62[m] = s62;
    }
    // fl32 of the top level: the ceil-absmax comparison value (its exponent is ohi)
    ft->lmax_mant = ft->dq_em[(1 << EC) - 1] & 0x7FFFFFu;
    ft->npoints = r.nmid;
    for (int i = 0; i < r.nmid; i++) {
        ft->point_o[i] = r.mid[i].o;
        ft->point_T[i] = r.mid[i].T;
    }
    ft->zero_o = r.zero.o;
    ft->zero_T = r.zero.T;
    ft->zero_exact = r.zero.exact ? 1 : 0;
    if ((int)((int32_t)ft->dq_em[(1 << EC) - 1] >> 24) != ohi) return false;
    // GEMM expansion pairs: value (-1)^s 2^{w + bias} 2^{f/N}, bias = 15 - ohi (the row's top
    // element lands near 2^15), hi = RN16(v), lo = RN16(v - hi)
    const int bias = 15 - ohi;
    memset(ft->dec, 0, sizeof(ft->dec));
    for (int code = 0; code < (1 << (EC + 1)); code++) {
        const int m = code & ((1 << EC) - 1);
        const int sgn = (code >> EC) & 1;
        if (m == 0) continue;
        const int u = P * (m - r.B);
        const int w = floor_div(u, N), f = u - w * N;
        long double v = ldexpl(pow2frac(f, N), w + bias);
        uint16_t hb, lb;
        if (!rn_fp16(v, &hb)) return false;
        long double rest = v - fp16_value(hb);
        if (!rn_fp16(fabsl(rest), &lb)) return false;
        if (lb && rest < 0) lb |= 0x8000;
        if (sgn) { hb ^= 0x8000; if (lb) lb ^= 0x8000; }
        ft->dec[code] = ((uint32_t)lb << 16) | hb;
    }
    return true;
}

}  // namespace

bool build_tables(AllTables* t) {
    static_assert(NUM_FORMATS == 5, "one builder call per format");
    return build_format(4, 3, 1, 1, &t->f[0]) && build_format(5, 2, 1, 1, &t->f[1]) &&
           build_format(3, 3, 1, 1, &t->f[2]) && build_format(4, 3, 8, 9, &t->f[3]) &&
           build_format(4, 3, 3, 4, &t->f[4]);
}

}  // namespace curvefp
