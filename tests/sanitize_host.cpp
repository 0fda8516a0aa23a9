// Host-side checks of the library's host code (moduli.cpp: moduli, roots, CRT
// weights, budgets) and of the header-only helpers the kernels share with the
// host (crt_round.h, tile_schedule.h, sym_schedule.h), built with
// AddressSanitizer and UndefinedBehaviorSanitizer by
// tests/test_host_sanitizers.py.  Output lines are compared there with the
// oracle and Python integers.
//
//   stdin:  "r T sc f32 c_0 ... c_{T-1}" lines: the limbs of an integer,
//           rounded once into fp64 (f32 = 0) or fp32 (f32 = 1) after 2^sc;
//           "b t S2 S1 n U" lines: one Cauchy-Schwarz chunk record one
//           binade count t below the row maximum, and a sum U (cs_bounds.h)
//   stdout: "r <bits of the double>" per r line, "b <lo> <hi> <d of U>" per b
//           line, then the moduli tables
//           ("m N log2M limbs P(k=1024) P(k=65536) cs_ok m_1 s_1 ... m_N s_N")
//           and "sched <shapes checked>" after the tile-schedule coverage
//           checks (which abort on a failure).
#define O2M_HD
#include <inttypes.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <vector>

#include "../paper_2609_05419_amd/csrc/crt_round.h"
#include "../paper_2609_05419_amd/csrc/cs_bounds.h"
#include "../paper_2609_05419_amd/csrc/o2m_internal.h"
#include "../paper_2609_05419_amd/csrc/sym_schedule.h"
#include "../paper_2609_05419_amd/csrc/tile_schedule.h"

namespace {

template <int W>
double round_limbs(const int64_t *c, int T, int sc, bool f32) {
    o2m::UW<W> v = {};
    for (int t = 0; t < T; ++t) o2m::add_shifted<W>(v, c[t], 40 * t);
    return f32 ? o2m::round_words_fmt<W, 24, -126>(v, sc) : o2m::round_words_fmt<W, 53, -1022>(v, sc);
}

void fail(const char *what, long a, long b) {
    fprintf(stderr, "FAIL %s %ld %ld\n", what, a, b);
    abort();
}

// every tile of every product exactly once over the fixed and pooled slots
long check_gemm_schedule(int mt, int nt, int kblocks, int batch) {
    const o2m::GemmSchedule s = o2m::gemm_schedule(mt, nt, kblocks, batch, o2m::kStageBytes);
    std::vector<int> seen((size_t)mt * nt * batch, 0);
    for (int x = 0; x < o2m::kXcds; ++x)
        for (long slot = 0; slot < s.slots; ++slot) {
            const o2m::TileCoord c = o2m::tile_of(x, (int)slot, mt, nt, s.chunk, s.deal);
            if (!c.valid) continue;
            if (c.p < 0 || c.p >= batch || c.ti < 0 || c.ti >= mt || c.tj < 0 || c.tj >= nt)
                fail("tile out of range", slot, x);
            seen[((size_t)c.p * mt + c.ti) * nt + c.tj]++;
        }
    for (size_t i = 0; i < seen.size(); ++i)
        if (seen[i] != 1) fail("tile count", (long)i, seen[i]);
    return (long)seen.size();
}

long check_sym_schedule(int nb) {
    const long grid = o2m::sym_grid(nb);
    std::vector<int> seen((size_t)nb * nb, 0);
    for (long b = 0; b < grid; ++b) {
        const o2m::SymTile t = o2m::sym_tile_of(b, nb);
        if (!t.valid) continue;
        if (t.I < 0 || t.I >= nb || t.J < 0 || t.J > t.I) fail("sym tile out of range", b, nb);
        seen[(size_t)t.I * nb + t.J]++;
    }
    for (int i = 0; i < nb; ++i)
        for (int j = 0; j <= i; ++j)
            if (seen[(size_t)i * nb + j] != 1) fail("sym tile count", i, j);
    return grid;
}

}  // namespace

int main() {
    char line[4096];
    while (fgets(line, sizeof line, stdin)) {
        if (line[0] == 'b') {
            int t = 0;
            uint64_t s2 = 0, s1 = 0, n = 0, U = 0, lo = 0, hi = 0;
            if (sscanf(line + 1, "%d %" SCNu64 " %" SCNu64 " %" SCNu64 " %" SCNu64, &t, &s2, &s1, &n, &U) != 5)
                fail("bad b line", t, 0);
            o2m::cs_chunk_bounds(t, s2, s1, n, &lo, &hi);
            printf("b %" PRIu64 " %" PRIu64 " %d\n", lo, hi, o2m::cs_d_of(U));
            continue;
        }
        if (line[0] != 'r') continue;
        int T = 0, sc = 0, f32 = 0, pos = 0;
        char *p = line + 1;
        if (sscanf(p, "%d %d %d%n", &T, &sc, &f32, &pos) != 3 || T < 1 || T > 6) fail("bad line", T, 0);
        p += pos;
        int64_t c[6] = {0, 0, 0, 0, 0, 0};
        for (int t = 0; t < T; ++t) {
            if (sscanf(p, "%" SCNd64 "%n", &c[t], &pos) != 1) fail("bad limb", t, 0);
            p += pos;
        }
        const double r = T <= 4 ? round_limbs<3>(c, T, sc, f32 != 0) : round_limbs<4>(c, T, sc, f32 != 0);
        uint64_t bits;
        memcpy(&bits, &r, sizeof bits);
        printf("r %016" PRIx64 "\n", bits);
    }
    for (int N = 1; N <= o2m::kMaxModuli; ++N) {
        const o2m::ModuliTable *t = o2m::moduli_table(N);
        int qa = 0, qb = 0;
        const bool cs = o2m::budget_cs(t, 8192, false, &qa, &qb);
        printf("m %d %.9f %d %d %d %d %d %d", N, t->log2M, t->crt.limbs, o2m::budget(t, 1024), o2m::budget(t, 65536),
               (int)cs, qa, qb);
        for (int l = 0; l < N; ++l) printf(" %d %d", t->res.mod[l], t->res.root[l]);
        printf("\n");
    }
    long checked = 0;
    const int shapes[][4] = {{1, 1, 1, 1}, {4, 4, 128, 32}, {32, 32, 128, 32}, {33, 17, 200, 5}, {64, 64, 256, 2},
                             {9, 40, 130, 44}, {7, 3, 1, 70}};
    for (const auto &s : shapes) checked += check_gemm_schedule(s[0], s[1], s[2], s[3]);
    for (int nb : {1, 2, 3, 5, 8, 13, 31, 64, 129}) checked += check_sym_schedule(nb);
    printf("sched %ld\n", checked);
    return 0;
}
