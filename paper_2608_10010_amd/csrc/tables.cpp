// Host construction of libcurvefp's constant tables.
//
// All irrational constants 2^{k/K} come from x87 80-bit exp2l (64-bit
// significand).  Every integer decision taken from them (a threshold floor, a
// rounding direction) is checked to sit far from the ambiguous point, so the
// 64-bit approximation cannot flip it; a failed check makes build_tables
// return false and the library refuses to run.
//
// Quantizer (Sec. 3.1): within an octave [2^o, 2^{o+1}) the levels are
// 2^{o + c/K}; the magnitude y = M 2^{o-23} (M the 24-bit significand) is
// nearest to 2^{o + c/K} with c = #{h : M > T_h}, T_h = floor(2^22 (2^{h/K} +
// 2^{(h+1)/K})) -- the midpoints are irrational, so no integer M sits on one.
// Below the smallest level the choice is between zero and 2^{n_min/K}, decided
// by the midpoint 2^{n_min/K - 1}.
#include <cmath>
#include <cstdio>
#include <cstring>

#include "curvefp_internal.hpp"

namespace curvefp {
namespace {

long double pow2frac(int k, int K) { return exp2l((long double)k / (long double)K); }

// floor(x) where x is known to lie far from an integer
bool safe_floor(long double x, int64_t* out) {
    long double f = floorl(x);
    long double fr = x - f;
    if (fr < 1e-7L || fr > 1.0L - 1e-7L) return false;
    *out = (int64_t)f;
    return true;
}

struct Rule {
    int K, B, nmin, nmax, oz;
    int64_t T[8];   // regular thresholds on the 24-bit significand
    int64_t Tz;     // zero threshold significand in octave oz
};

bool make_rule(int E, int C, Rule* r) {
    r->K = 1 << C;
    r->B = 1 << (E + C - 1);
    r->nmin = -(r->B - 1);
    r->nmax = r->B - 1;
    const int K = r->K;
    for (int h = 0; h < K; h++) {
        long double t = ldexpl(pow2frac(h, K) + pow2frac(h + 1, K), 22);
        if (!safe_floor(t, &r->T[h])) return false;
    }
    // 2^{n_min/K - 1} = 2^{oz} * 2^{rem/K}, rem in [0, K)
    int num = r->nmin - K;
    int oz = num >= 0 ? num / K : -((-num + K - 1) / K);
    int rem = num - oz * K;
    r->oz = oz;
    if (rem == 0) return false;  // would be a representable (tie-able) threshold
    if (!safe_floor(ldexpl(pow2frac(rem, K), 23), &r->Tz)) return false;
    return true;
}

// magnitude rank (0 = zero) of y = M 2^{o - 23}
int rank_of(const Rule& r, int o, int64_t M) {
    int c = 0;
    for (int h = 0; h < r.K; h++) c += (M > r.T[h]);
    int n = r.K * o + c;
    if (n > r.nmax) n = r.nmax;
    if (n < r.nmin) {
        bool above = (o > r.oz) || (o == r.oz && M > r.Tz);
        if (!above) return 0;
        n = r.nmin;
    }
    return n + r.B;
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

bool build_format(int E, int C, FormatTables* ft) {
    Rule r;
    if (!make_rule(E, C, &r)) return false;
    const int K = r.K;
    ft->K = K;
    const int ohi = r.nmax / K;
    ft->qlut_size = (ohi - r.oz + 1) * 128;
    if (ft->qlut_size > QLUT_MAX) return false;
    for (int i = 0; i < ft->qlut_size; i++) {
        int o = r.oz + i / 128;
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
    // fl32(2^{k/K}) mantissas and 62-bit significands
    for (int k = 0; k < 8; k++) { ft->mant[k] = 0; ft->sig62[k] = 0; }
    for (int k = 0; k < K; k++) {
        long double s = pow2frac(k, K);
        long double q = ldexpl(s, 23);
        long double fl = floorl(q), fr = q - fl;
        if (k && fabsl(fr - 0.5L) < 1e-9L) return false;
        uint32_t qi = (uint32_t)fl + (fr > 0.5L ? 1u : 0u);
        if (qi >= (1u << 24)) return false;
        ft->mant[k] = qi - (1u << 23);
        long double q62 = ldexpl(s, 62);
        ft->sig62[k] = (uint64_t)floorl(q62);
        // the subnormal reconstruction rounds sig62 at bit positions 40..63
        for (int sh = 40; sh <= 63 && k; sh++) {
            uint64_t rem = ft->sig62[k] & ((1ull << sh) - 1);
            uint64_t half = 1ull << (sh - 1);
            uint64_t d = rem > half ? rem - half : half - rem;
            if (d < 4) return false;
        }
    }
    ft->lmax_mant = ft->mant[K - 1];
    // GEMM expansion pairs: value (-1)^s 2^{e + bias} 2^{k/K}, hi = RN16(v), lo = RN16(v - hi)
    const int EMAX = (1 << (E - 1)) - 1;
    const int bias = 15 - EMAX;
    const int EC = E + C;
    memset(ft->dec, 0, sizeof(ft->dec));
    for (int code = 0; code < (1 << (EC + 1)); code++) {
        const int m = code & ((1 << EC) - 1);
        const int sgn = (code >> EC) & 1;
        if (m == 0) continue;
        int n = m - r.B;
        int e = (n >= 0) ? n / K : -((-n + K - 1) / K);
        int k = n - e * K;
        long double v = ldexpl(pow2frac(k, K), e + bias);
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
    return build_format(4, 3, &t->f[0]) && build_format(5, 2, &t->f[1]) && build_format(3, 3, &t->f[2]);
}

}  // namespace curvefp
