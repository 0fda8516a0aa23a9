// Exact CRT lift and correct rounding, shared by the CRT kernels and the
// host-compiled unit test of this header.  Host and device code see the same
// source; nothing here touches memory.
//
// The lifted CRT value (Algorithm 1, step 6) is an integer c held as T limbs,
// c = sum_t c_t 2^(40 t), each limb an integer-valued double with |c_t| < 2^53.
// Step 7 needs RN(c) (round to nearest, ties to even), then a scaling by 2^sc.
#pragma once

#include <math.h>
#include <stdint.h>

#ifndef O2M_HD
#define O2M_HD __host__ __device__
#endif

namespace o2m {

constexpr double kTwo40 = 1099511627776.0;
constexpr double kTwo80 = 1208925819614629174706176.0;

O2M_HD inline int64_t bits_of_f64(double x) { return __builtin_bit_cast(int64_t, x); }
O2M_HD inline double f64_of_bits(int64_t b) { return __builtin_bit_cast(double, b); }

// Knuth's TwoSum: s = RN(a + b) and e = (a + b) - s exactly.
O2M_HD inline void two_sum(double a, double b, double &s, double &e) {
    s = a + b;
    const double bb = s - a;
    e = (a - (s - bb)) + (b - bb);
}

// x + y rounded to odd: the exact sum if representable, otherwise the one of
// its two neighbouring doubles whose last significand bit is 1.
O2M_HD inline double sum_round_odd(double x, double y) {
    double s, e;
    two_sum(x, y, s, e);
    if (e != 0.0) {
        int64_t b = bits_of_f64(s);
        if ((b & 1) == 0) b += ((e > 0.0) == (s > 0.0)) ? 1 : -1;  // step toward e
        s = f64_of_bits(b);
    }
    return s;
}

// RN(a + b + c) for any doubles without overflow or underflow (Boldo and
// Melquiond, correctly rounded sum of three numbers via rounding to odd):
// (uh, ul) = TwoSum(b, c), (th, tl) = TwoSum(a, uh), RN(th + RO(tl + ul)).
O2M_HD inline double sum3_rn(double a, double b, double c) {
    double uh, ul, th, tl;
    two_sum(b, c, uh, ul);
    two_sum(a, uh, th, tl);
    return th + sum_round_odd(tl, ul);
}

// Two's complement integer of W 64-bit words, little-endian.
template <int W>
struct UW {
    uint64_t w[W];
};

// a += x * 2^s (modulo 2^(64 W)); 0 <= s < 64 (W - 1).
template <int W>
O2M_HD inline void add_shifted(UW<W> &a, int64_t x, int s) {
    const uint64_t ux = (uint64_t)x;
    const uint64_t ext = (uint64_t)(x >> 63);
    const int ws = s >> 6, bs = s & 63;
    uint64_t carry = 0;
#pragma unroll
    for (int i = 0; i < W; ++i) {
        uint64_t y;
        if (i < ws) y = 0;
        else if (i == ws) y = ux << bs;
        else if (i == ws + 1) y = bs ? (ux >> (64 - bs)) | (ext << bs) : ext;
        else y = ext;
        const uint64_t t = a.w[i] + y;
        const uint64_t c1 = t < y;
        const uint64_t r = t + carry;
        const uint64_t c2 = r < carry;
        a.w[i] = r;
        carry = c1 + c2;
    }
}

O2M_HD inline int clz64(uint64_t x) { return __builtin_clzll(x); }

// RN of a W-word signed integer, ties to even, times 2^sc (one rounding).
template <int W>
O2M_HD inline double round_words(UW<W> v, int sc) {
    const bool neg = (int64_t)v.w[W - 1] < 0;
    if (neg) {
        uint64_t carry = 1;
#pragma unroll
        for (int i = 0; i < W; ++i) {
            const uint64_t t = ~v.w[i] + carry;
            carry = carry && t == 0;
            v.w[i] = t;
        }
    }
    // the most significant nonzero word (hi), the word below it (lo) and the
    // OR of all lower words; every index is static, so the words stay in
    // registers
    int top = -1;
    uint64_t hi = 0, lo = 0, low = 0;
#pragma unroll
    for (int i = W - 1; i >= 0; --i) {
        if (top < 0 && v.w[i] != 0) {
            top = i;
            hi = v.w[i];
            lo = i > 0 ? v.w[i > 0 ? i - 1 : 0] : 0;
        }
    }
    if (top < 0) return 0.0;
#pragma unroll
    for (int i = 0; i + 2 < W; ++i)
        if (i < top - 1) low |= v.w[i];
    const int lz = clz64(hi);
    // h = the 64 bits below the leading one (inclusive), rest = sticky bits
    uint64_t h = hi << lz;
    if (lz) h |= lo >> (64 - lz);
    const uint64_t rest = (lo << lz) | low;
    uint64_t mant = h >> 11;
    const uint64_t rb = h & 0x7FF;
    if (rb > 0x400 || (rb == 0x400 && (rest != 0 || (mant & 1)))) mant += 1;
    const int msb = 64 * top + 63 - lz;  // bit index of the leading one
    const double r = ldexp((double)mant, msb - 52 + sc);
    return neg ? -r : r;
}

// Words needed for T limbs of 40 bits with |c_t| < 2^53, plus the sign.
template <int T>
struct LimbWords {
    static constexpr int value = (40 * (T - 1) + 54 + 63) / 64;
};

// Steps 5-7 for one component: limb sums S_t = sum_l u_l w_lt (exact), the
// quotient q = rint(X / M) from a fp64 Horner sum (exact while |c| / M stays
// below 1/2 - 2^-32), the lifted limbs c_t = S_t - q M_t (exact), and
// RN(c) * 2^sc.  T <= 3 rounds with the three-term sum; T >= 4 through a
// multiword integer (192 bits for T = 4, 256 bits for T = 5, 6).
template <int T>
O2M_HD inline double lift_round(const double (&S)[T], const double *mlimb, double inv_m, int sc) {
    double X = S[T - 1];
    for (int t = T - 2; t >= 0; --t) X = fma(X, kTwo40, S[t]);
    const double q = rint(X * inv_m);
    double c[T];
    for (int t = 0; t < T; ++t) c[t] = fma(-q, mlimb[t], S[t]);
    if constexpr (T == 2) {
        return ldexp(fma(c[1], kTwo40, c[0]), sc);              // one rounding of an exact sum
    } else if constexpr (T == 3) {
        return ldexp(sum3_rn(c[2] * kTwo80, c[1] * kTwo40, c[0]), sc);
    } else {
        constexpr int W = LimbWords<T>::value;
        UW<W> v = {};
#pragma unroll
        for (int t = 0; t < T; ++t) add_shifted<W>(v, (int64_t)c[t], 40 * t);
        return round_words<W>(v, sc);
    }
}

// The exact lifted integer (Gaussian-integer mode: M < 2^63, two limbs).
template <int T>
O2M_HD inline UW<LimbWords<T>::value> lift_exact(const double (&S)[T], const double *mlimb, double inv_m) {
    double X = S[T - 1];
    for (int t = T - 2; t >= 0; --t) X = fma(X, kTwo40, S[t]);
    const double q = rint(X * inv_m);
    constexpr int W = LimbWords<T>::value;
    UW<W> v = {};
#pragma unroll
    for (int t = 0; t < T; ++t) add_shifted<W>(v, (int64_t)fma(-q, mlimb[t], S[t]), 40 * t);
    return v;
}

}  // namespace o2m
