// Host build of the one-pass Cauchy-Schwarz helpers (cs_bounds.h), for
// tests/test_cs_bounds.py.
#define O2M_HD
#include "../paper_2609_05419_amd/csrc/cs_bounds.h"

extern "C" {
int t_cs_d_of(uint64_t U) { return o2m::cs_d_of(U); }
void t_cs_chunk_bounds(int t, uint64_t s2, uint64_t s1, uint64_t n, uint64_t *lo, uint64_t *hi) {
    o2m::cs_chunk_bounds(t, s2, s1, n, lo, hi);
}
}
