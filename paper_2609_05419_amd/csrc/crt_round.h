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

// 192-bit two's complement integer, little-endian 64-bit words.
struct U192 {
    uint64_t w0, w1, w2;
};

// a += x * 2^s (modulo 2^192); s is a multiple of 40 below 192.
O2M_HD inline void add_shifted(U192 &a, int64_t x, int s) {
    const uint64_t ux = (uint64_t)x;
    const uint64_t ext = (uint64_t)(x >> 63);
    uint64_t y0, y1, y2;
    if (s == 0) {
        y0 = ux; y1 = ext; y2 = ext;
    } else if (s < 64) {
        y0 = ux << s; y1 = (ux >> (64 - s)) | (ext << s); y2 = ext;
    } else if (s < 128) {
        const int t = s - 64;
        y0 = 0; y1 = ux << t; y2 = (ux >> (64 - t)) | (ext << t);
    } else {
        y0 = 0; y1 = 0; y2 = ux << (s - 128);
    }
    const uint64_t r0 = a.w0 + y0;
    const uint64_t c0 = r0 < y0;
    uint64_t r1 = a.w1 + y1;
    uint64_t c1 = r1 < y1;
    r1 += c0;
    c1 += r1 < c0;
    a.w0 = r0;
    a.w1 = r1;
    a.w2 = a.w2 + y2 + c1;
}

O2M_HD inline int clz64(uint64_t x) { return __builtin_clzll(x); }

// RN of a 192-bit signed integer, ties to even, times 2^sc (one rounding).
O2M_HD inline double round_u192(U192 v, int sc) {
    const bool neg = (int64_t)v.w2 < 0;
    if (neg) {
        v.w0 = ~v.w0; v.w1 = ~v.w1; v.w2 = ~v.w2;
        v.w0 += 1;
        const uint64_t c0 = v.w0 == 0;
        v.w1 += c0;
        v.w2 += (c0 && v.w1 == 0);
    }
    int lz;
    if (v.w2) lz = clz64(v.w2);
    else if (v.w1) lz = 64 + clz64(v.w1);
    else if (v.w0) lz = 128 + clz64(v.w0);
    else return 0.0;
    uint64_t h, rest;
    if (lz >= 128) {
        h = v.w0 << (lz - 128);
        rest = 0;
    } else if (lz >= 64) {
        const int s = lz - 64;
        h = s ? (v.w1 << s) | (v.w0 >> (64 - s)) : v.w1;
        rest = s ? (v.w0 << s) : v.w0;
    } else {
        const int s = lz;
        h = s ? (v.w2 << s) | (v.w1 >> (64 - s)) : v.w2;
        const uint64_t n1 = s ? (v.w1 << s) | (v.w0 >> (64 - s)) : v.w1;
        const uint64_t n0 = s ? (v.w0 << s) : v.w0;
        rest = n1 | n0;
    }
    uint64_t mant = h >> 11;
    const uint64_t rb = h & 0x7FF;
    if (rb > 0x400 || (rb == 0x400 && (rest != 0 || (mant & 1)))) mant += 1;
    const int top = 191 - lz;
    const double r = ldexp((double)mant, top - 52 + sc);
    return neg ? -r : r;
}

// Steps 5-7 for one component: limb sums S_t = sum_l u_l w_lt (exact), the
// quotient q = rint(X / M) from a fp64 Horner sum (exact while |c| / M stays
// below 1/2 - 2^-32), the lifted limbs c_t = S_t - q M_t (exact), and
// RN(c) * 2^sc.  T <= 3 rounds with the three-term sum; T = 4 through a
// 192-bit integer.
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
        U192 v = {0, 0, 0};
        for (int t = 0; t < T; ++t) add_shifted(v, (int64_t)c[t], 40 * t);
        return round_u192(v, sc);
    }
}

// The exact lifted integer as 192 bits (Gaussian-integer mode).
template <int T>
O2M_HD inline U192 lift_exact(const double (&S)[T], const double *mlimb, double inv_m) {
    double X = S[T - 1];
    for (int t = T - 2; t >= 0; --t) X = fma(X, kTwo40, S[t]);
    const double q = rint(X * inv_m);
    U192 v = {0, 0, 0};
    for (int t = 0; t < T; ++t) add_shifted(v, (int64_t)fma(-q, mlimb[t], S[t]), 40 * t);
    return v;
}

}  // namespace o2m
