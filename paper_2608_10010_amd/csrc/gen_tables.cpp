// Build-time generator of libcurvefp's constant tables.
//
//   gen_tables OUT.inc      writes the tables as C initializer macros; the kernel sources include
//                           the file and hold every table as a __constant__ array, so the library
//                           needs no upload, no per-device state and no synchronization
//   gen_tables --report     prints each format's decision points (the nearest-level rule's
//                           thresholds, Sec. 3.1) for the host tests
//
// The derivation itself (x87 exp2l, every integer decision checked far from its ambiguous point)
// is tables.cpp's; if one of its checks fails the generator exits with status 1 and the build
// stops.
#include <cinttypes>
#include <cstdio>
#include <cstring>
#include <string>

#include "tables.hpp"

using namespace curvefp;

namespace {

const char* kNames[NUM_FORMATS] = {"E4C3", "E5C2", "E3C3", "E4C3_r8/9", "E4C3_r3/4"};

// one "{a, b, ...}" row per format; get(f, i) gives entry i of format f
template <class G>
void table(FILE* out, const char* name, int n, const char* fmt, G get) {
    fprintf(out, "#define %s { \\\n", name);
    for (int f = 0; f < NUM_FORMATS; f++) {
        fprintf(out, "  {");
        for (int i = 0; i < n; i++) {
            if (i % 8 == 0) fprintf(out, " \\\n   ");
            fprintf(out, fmt, get(f, i));
            fprintf(out, "%s", i + 1 < n ? ", " : "");
        }
        fprintf(out, "}%s \\\n", f + 1 < NUM_FORMATS ? "," : "");
    }
    fprintf(out, "}\n\n");
}

int write_inc(const AllTables& t, const char* path) {
    FILE* out = fopen(path, "w");
    if (!out) {
        perror(path);
        return 1;
    }
    fprintf(out, "// Constant tables of libcurvefp, written at build time by gen_tables (derivation in\n"
                 "// tables.cpp).  Do not edit.  One row per format id of the C ABI.\n#pragma once\n\n");
    auto bin = [&](int f) { return t.f[f].P == 1 && t.f[f].Q == 1; };
    // quantizer: (base rank << 16) | 16-bit threshold per bf16-truncated magnitude bucket, and
    // the base rank alone (bf16 sources)
    table(out, "CURVEFP_QLUT_INIT", QLUT_MAX, "0x%08" PRIx32 "u", [&](int f, int i) { return t.f[f].qlut[i]; });
    table(out, "CURVEFP_QLUT8_INIT", QLUT_MAX, "%" PRIu32 "u",
          [&](int f, int i) { return (uint32_t)(uint8_t)(t.f[f].qlut[i] >> 16); });
    // reconstruction: binary radix by curve index (8 entries), rational radix by magnitude rank
    table(out, "CURVEFP_MANT_INIT", 8, "0x%06" PRIx32 "u", [&](int f, int i) { return t.f[f].mant[i]; });
    table(out, "CURVEFP_SIG62_INIT", 8, "0x%016" PRIx64 "ull", [&](int f, int i) { return t.f[f].sig62[i]; });
    table(out, "CURVEFP_DQ_EM_INIT", 128, "0x%08" PRIx32 "u", [&](int f, int i) { return t.f[f].dq_em[i]; });
    table(out, "CURVEFP_DQ_SIG62_INIT", 128, "0x%016" PRIx64 "ull",
          [&](int f, int i) { return t.f[f].dq_sig62[i]; });
    // the static-scale search's reconstruction table: the binary or the rational one, by format
    table(out, "CURVEFP_QR_MANT_INIT", 128, "0x%08" PRIx32 "u", [&](int f, int i) {
        return bin(f) ? (i < 8 ? t.f[f].mant[i] : 0u) : t.f[f].dq_em[i];
    });
    table(out, "CURVEFP_QR_SIG_INIT", 128, "0x%016" PRIx64 "ull", [&](int f, int i) {
        return bin(f) ? (i < 8 ? t.f[f].sig62[i] : 0ull) : t.f[f].dq_sig62[i];
    });
    // GEMM expansion: (lo16 << 16) | hi16 fp16 pair per code byte
    table(out, "CURVEFP_DEC_INIT", GEMM_DEC_ENTRIES, "0x%08" PRIx32 "u", [&](int f, int i) { return t.f[f].dec[i]; });
    // per format: the mantissa field of fl32 of the top level (the ceil-absmax comparison value),
    // and the quantizer table's size
    fprintf(out, "#define CURVEFP_LMAX_MANT_INIT {");
    for (int f = 0; f < NUM_FORMATS; f++) fprintf(out, "0x%06" PRIx32 "u%s", t.f[f].lmax_mant, f + 1 < NUM_FORMATS ? ", " : "");
    fprintf(out, "}\n");
    fprintf(out, "#define CURVEFP_QLUT_SIZE_INIT {");
    for (int f = 0; f < NUM_FORMATS; f++) fprintf(out, "%d%s", t.f[f].qlut_size, f + 1 < NUM_FORMATS ? ", " : "");
    fprintf(out, "}\n");
    if (fclose(out) != 0) {
        perror(path);
        return 1;
    }
    return 0;
}

void report(const AllTables& t) {
    for (int f = 0; f < NUM_FORMATS; f++) {
        const FormatTables& ft = t.f[f];
        printf("format %d %s K=%d P=%d Q=%d qlut=%d lmax_mant=0x%06" PRIx32 "\n", f, kNames[f], ft.K, ft.P, ft.Q,
               ft.qlut_size, ft.lmax_mant);
        printf("zero %d %" PRId64 " %d\n", ft.zero_o, ft.zero_T, ft.zero_exact);
        for (int i = 0; i < ft.npoints; i++) printf("mid %d %d %" PRId64 "\n", i, ft.point_o[i], ft.point_T[i]);
        for (int m = 0; m < 128; m++) printf("dq_em %d 0x%08" PRIx32 "\n", m, ft.dq_em[m]);
        for (int c = 0; c < GEMM_DEC_ENTRIES; c++) printf("dec %d 0x%08" PRIx32 "\n", c, ft.dec[c]);
    }
}

}  // namespace

int main(int argc, char** argv) {
    if (argc != 2) {
        fprintf(stderr, "usage: gen_tables OUT.inc | --report\n");
        return 2;
    }
    static AllTables t;
    if (!build_tables(&t)) {
        fprintf(stderr, "gen_tables: a self-check of the table derivation failed\n");
        return 1;
    }
    if (std::string(argv[1]) == "--report") {
        report(t);
        return 0;
    }
    return write_inc(t, argv[1]);
}
