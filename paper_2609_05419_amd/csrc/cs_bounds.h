// Cauchy-Schwarz exponents from one pass over an operand (K1).
//
// The rule (a norm-based choice of the power-of-two scales sigma, tau, which
// Section 3.1 leaves to the Ozaki-II literature) bounds the 2-norm of a row by
// 2^G with G = E - 20 + d, where E is the row's max exponent (every part
// |v| < 2^E), d the least d >= 0 with 4^d >= U, and
//     U = sum over the nonzero parts v of the row of max(1, ceil(|v| 2^(20 - E)))^2,
// an exact integer.  U needs E, which a single pass does not know yet.  The
// pass therefore reduces each chunk of the row against the chunk's own max
// exponent e <= E: with y = max(1, ceil(|v| 2^(20 - e))) it keeps
//     S2 = sum y^2,  S1 = sum y,  n = number of nonzero parts,
// and since ceil(y / 2^t) = ceil(|v| 2^(20 - E)) for t = E - e (ceil(x / q) =
// ceil(ceil(x) / q) for an integer q >= 1), each chunk's exact share of U lies in
//     [ max(n, ceil(S2 / 4^t)),  min(n 4^(20 - t), floor((S2 + 2 (2^t - 1) S1 + (2^t - 1)^2 n) / 4^t)) ]
// (y/q <= ceil(y/q) <= (y + q - 1)/q and 1 <= ceil(y/q) <= 2^(20 - t)), which is
// exact for t = 0 and, since every y <= 2^20, for t >= 21 (each term is 1).
// When both ends of the summed interval give the same d the exponent is
// exact; otherwise the row is marked and its U recomputed from the data.
// Shared by the kernels and by host tests.
#pragma once
#include <stdint.h>

#ifndef O2M_HD
#define O2M_HD __host__ __device__
#endif

namespace o2m {

// d = the least d >= 0 with 4^d >= U (0 for U <= 1).
O2M_HD inline int cs_d_of(uint64_t U) {
    if (U <= 1) return 0;
    const int bits = 64 - __builtin_clzll(U - 1);  // bit length of U - 1
    return (bits + 1) / 2;
}

// Interval [lo, hi] holding one chunk's exact share of U (see above);
// t = E - e >= 0.
O2M_HD inline void cs_chunk_bounds(int t, uint64_t s2, uint64_t s1, uint64_t n, uint64_t *lo, uint64_t *hi) {
    if (n == 0) {
        *lo = *hi = 0;
    } else if (t == 0) {
        *lo = *hi = s2;
    } else if (t >= 21) {
        *lo = *hi = n;
    } else {
        const uint64_t q = 1ull << t, q2 = 1ull << (2 * t);
        uint64_t l = (s2 + q2 - 1) >> (2 * t);
        if (l < n) l = n;
        uint64_t h = (s2 + 2 * (q - 1) * s1 + (q - 1) * (q - 1) * n) >> (2 * t);
        const uint64_t cap = n << (2 * (20 - t));
        if (h > cap) h = cap;
        *lo = l;
        *hi = h;
    }
}

}  // namespace o2m
