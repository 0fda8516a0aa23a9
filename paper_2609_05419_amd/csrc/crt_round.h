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
constexpr double kTwo120 = 1329227995784915872903807060280344576.0;

// A constant held in scalar registers on the device: a literal operand only
// fits the two-operand fma, which costs a register copy whenever its addend
// is still needed, while a scalar-register operand fits the three-operand
// form.  The empty asm only pins the value there; it emits no instruction.
O2M_HD inline double in_sreg(double x) {
#ifdef __HIP_DEVICE_COMPILE__
    asm("" : "+s"(x));
#endif
    return x;
}

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

// RN(a + b + y) for three terms split on a base-2^40 digit boundary: a and
// b integer multiples of 2^G (G = 40 (j - 1)), a = 0 or |a| >= 2^(G + 40) >
// 2^(G + 39) >= |b|, and y = 0 or 0 < |y| < 2^G, given as y itself when a
// double holds it (always when a = 0) or else rounded to odd.  s = RN(a + b)
// has the exact error e = (a + b) - s (fast two-sum: |a| >= |b|, or a = 0
// and e = 0), a multiple of 2^G.  If e = 0, a + b + y rounds like s + y:
// with a != 0, |s| >= 2^(G + 39), so the doubles and midpoints near s + y
// are multiples of 2^(G - 15), doubles of y's scale (|y| < 2^G) with an
// even last bit, which y rounded to odd is not, and it lies on the same
// side of each of them as y.
// If e != 0, a + b was not a double, so the doubles next to s are at least
// 2^(G + 1) apart and |e| + |y| stays below half a gap unless a + b was
// exactly halfway (|e| half the gap on e's side): then y decides, and the
// result is the neighbour s + 2e when y points past the midpoint (e y > 0),
// else s.  |e| is half the gap exactly when s + 2e is a double, i.e. when
// RN(s + 2e) - s == 2e (otherwise s + 2e lies strictly between s and the
// neighbour).
O2M_HD inline double round_top3(double a, double b, double y) {
    const double s = a + b;
    const double e = b - (s - a);
    const double n = fma(2.0, e, s);
    if (n - s == 2.0 * e && e * y > 0.0) return n;
    return e == 0.0 ? s + y : s;
}

// RN(c2 2^80 + c1 2^40 + c0) for integer-valued limbs with |c_t| < 2^52.4
// (the lifted limbs of a three-limb CRT value: limb sums below 2^52 minus
// q M_t with |q| < 2^11.4 and |M_t| <= 2^39).  The two low limbs are carried
// into balanced digits d1, d0 (|d| <= 2^39, every step exact), and
// c = c2' 2^80 + d1 2^40 + d0 is rounded as in round_top3 (G = 40, y = d0),
// except that s + d0 needs no guard for e != 0: then the gaps next to s are
// at least 2^41 on e's side and 2^40 on the other, so s + d0 rounds to s
// (at |d0| = 2^39 below a power of two, a tie that goes to s, whose
// significand is even).
O2M_HD inline double round3_rn(double c0, double c1, double c2) {
    const double two40 = in_sreg(kTwo40);
    const double h0 = rint(c0 * 0x1p-40);
    const double d0 = fma(-h0, two40, c0);
    c1 += h0;
    const double h1 = rint(c1 * 0x1p-40);
    const double d1 = fma(-h1, two40, c1);
    c2 += h1;
    const double a = c2 * in_sreg(kTwo80);
    const double s = fma(d1, two40, a);
    const double e = fma(d1, two40, -(s - a));
    const double n = fma(2.0, e, s);
    return n - s == 2.0 * e && e * d0 > 0.0 ? n : s + d0;
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

// x + y + z rounded to odd (the same TwoSum cascade as sum3_rn with the last
// addition rounded to odd too).  The inner round-to-odd sum v of the two error
// terms has a last significand bit of 1 unless it is exact, so it is never a
// point of the outer sum's grid (multiples of half an ulp of th, all of them
// representable at v's smaller scale with an even last bit); th + v and the
// exact sum therefore lie strictly between the same two neighbouring doubles,
// or are both exact, and round to odd alike.
O2M_HD inline double sum3_ro(double a, double b, double c) {
    double uh, ul, th, tl;
    two_sum(b, c, uh, ul);
    two_sum(a, uh, th, tl);
    return sum_round_odd(th, sum_round_odd(tl, ul));
}

// The integer v of W words times 2^sc, rounded once to nearest (ties to even)
// into a binary format with P significand bits and least normal exponent EMIN
// (fp64: 53, -1022; fp32: 24, -126), subnormal results included.  The result
// is returned as a double holding the rounded value exactly (for fp32 it then
// narrows to float without a second rounding, or to an infinity beyond the
// fp32 range).  Zero gives +0; a negative value that rounds to zero gives -0.
template <int W, int P, int EMIN>
O2M_HD inline double round_words_fmt(UW<W> v, int sc) {
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
    const int e = 64 * top + 63 - lz + sc;   // the value lies in [2^e, 2^(e+1))
    // significand bits kept: P, fewer for a subnormal result
    const int keep = e >= EMIN ? P : P - (EMIN - e);
    double r;
    if (keep <= 0) {
        // below the least subnormal q = 2^(EMIN - P + 1): the value is in
        // [q/2, q) when keep == 0 (up unless exactly q/2, a tie to 0), else
        // below q/2
        r = keep == 0 && ((h << 1) != 0 || rest != 0) ? ldexp(1.0, EMIN - P + 1) : 0.0;
    } else {
        uint64_t mant = h >> (64 - keep);
        const uint64_t below = h << keep;   // the dropped bits of h, left aligned
        const bool half = (below >> 63) != 0;
        const bool sticky = (below << 1) != 0 || rest != 0;
        if (half && (sticky || (mant & 1))) mant += 1;  // may reach 2^keep: still exact
        r = ldexp((double)mant, e - keep + 1);
    }
    return neg ? -r : r;
}

// RN to fp64 of a W-word signed integer times 2^sc (one rounding).
template <int W>
O2M_HD inline double round_words(UW<W> v, int sc) {
    return round_words_fmt<W, 53, -1022>(v, sc);
}

// Words needed for T limbs of 40 bits with |c_t| < 2^53, plus the sign.
template <int T>
struct LimbWords {
    static constexpr int value = (40 * (T - 1) + 54 + 63) / 64;
};

// Step 6 for one component: the quotient q = rint(X / M) from a fp64 Horner
// sum of the limb sums S_t (exact while |c| / M stays below 1/2 - 2^-32) and
// the lifted limbs c_t = S_t - q M_t (exact).
template <int T>
O2M_HD inline void lift_limbs(const double (&S)[T], const double *mlimb, double inv_m, double (&c)[T]) {
    const double two40 = in_sreg(kTwo40);
    double X = S[T - 1];
    for (int t = T - 2; t >= 0; --t) X = fma(X, two40, S[t]);
    const double q = rint(X * inv_m);
    for (int t = 0; t < T; ++t) c[t] = fma(-q, mlimb[t], S[t]);
}

// The lifted limbs as one multiword integer.
template <int T>
O2M_HD inline UW<LimbWords<T>::value> words_of(const double (&c)[T]) {
    constexpr int W = LimbWords<T>::value;
    UW<W> v = {};
#pragma unroll
    for (int t = 0; t < T; ++t) add_shifted<W>(v, (int64_t)c[t], 40 * t);
    return v;
}

constexpr double kTwo160 = 1461501637330902918203684832716283019655932542976.0;
constexpr double kTwo200 = 1606938044258990275541962092341162602522202993782792835301376.0;

// Lifted limbs (|c_t| < 2^53, T = 4..6) as three terms a, b, low whose sum
// rounds like c, to nearest and to odd.  The limbs are first carry-normalized
// into balanced base-2^40 digits d_0..d_{T-1} (|d_t| <= 2^39 below the top
// one; every step exact in fp64).  With j the index of the top nonzero digit,
// a = d_j 2^(40 j), b = d_{j-1} 2^(40 (j-1)) and low = the sum y of the lower
// digits rounded to odd (exact when j <= 2: low = d_0).  For j >= 3,
// |c| > 2^(40 j - 2), so every double near c and every midpoint between two
// is a multiple of 2^(40 j - 55), and so is its distance from a + b (a
// multiple of 2^(40 j - 40)).  |y| < 2^(40 j - 40) makes the doubles of y's
// scale at most 2^(40 j - 93) apart, so such a multiple is a double of y's
// scale with an even last bit: RO(y), odd unless it equals y, lies on the
// same side of it as y.  Any rounding of a + b + low to nearest or to odd
// thus equals that of c.  RO(y) itself: the exact three-term sum rounded to
// odd for three digits, and for four digits the same construction one level
// down (their top digit weighs 2^120, where the margin is 2^38 again).
O2M_HD inline double ro_digits3(double d0, double d1, double d2) { return sum3_ro(d2 * kTwo80, d1 * kTwo40, d0); }

O2M_HD inline double ro_digits4(double d0, double d1, double d2, double d3) {
    return d3 != 0.0 ? sum3_ro(d3 * kTwo120, d2 * kTwo80, sum_round_odd(d1 * kTwo40, d0)) : ro_digits3(d0, d1, d2);
}

template <int T>
O2M_HD inline void top3_of(double (&c)[T], double &a, double &b, double &low) {
    static_assert(T >= 4 && T <= 6, "three-term reduction for four to six limbs");
    const double two40 = in_sreg(kTwo40);
#pragma unroll
    for (int t = 0; t + 1 < T; ++t) {
        const double h = rint(c[t] * (1.0 / kTwo40));
        c[t] = fma(-h, two40, c[t]);
        c[t + 1] += h;
    }
    if constexpr (T == 6) {
        if (c[5] != 0.0) {
            a = c[5] * kTwo200;
            b = c[4] * kTwo160;
            low = ro_digits4(c[0], c[1], c[2], c[3]);
            return;
        }
    }
    if constexpr (T >= 5) {
        if (c[4] != 0.0) {
            a = c[4] * kTwo160;
            b = c[3] * kTwo120;
            low = ro_digits3(c[0], c[1], c[2]);
            return;
        }
    }
    if (c[3] != 0.0) {
        a = c[3] * kTwo120;
        b = c[2] * kTwo80;
        low = sum_round_odd(c[1] * kTwo40, c[0]);
    } else {
        a = c[2] * kTwo80;
        b = c[1] * kTwo40;
        low = c[0];
    }
}

// Steps 5-7 for one component with fp64 output: the lifted limbs, then
// RN(c 2^sc), one rounding.  c is rounded with the exact limb sum (T = 2),
// round3_rn (T = 3) or round_top3 of top3_of's terms (T >= 4) and scaled by
// 2^sc,
// which is exact unless the result is subnormal; such results (and those that
// underflow to zero) are rounded again from the exact integer, held as 192 or
// 256 bits, at the subnormal quantum.  A value just below 2^-1022 can round
// to 2^-1022 itself in the scaling (the 53-bit value ties on the subnormal
// grid), so |r| = 2^-1022 takes the exact path too; rounding is monotone, so
// every exact value below 2^-1022 gives |r| <= 2^-1022.
template <int T>
O2M_HD inline double lift_round(const double (&S)[T], const double *mlimb, double inv_m, int sc) {
    double c[T];
    lift_limbs<T>(S, mlimb, inv_m, c);
    double x;
    if constexpr (T == 2) {
        x = fma(c[1], in_sreg(kTwo40), c[0]);     // one rounding of an exact sum
    } else if constexpr (T == 3) {
        x = round3_rn(c[0], c[1], c[2]);
    } else {
        double a, b, low;
        top3_of<T>(c, a, b, low);
        x = round_top3(a, b, low);
    }
    const double r = ldexp(x, sc);
    if (x == 0.0 || !(fabs(r) <= 0x1p-1022)) return r;
    return round_words<LimbWords<T>::value>(words_of<T>(c), sc);
}

// Steps 5-7 with fp32 output (CGEMM): RN32(c 2^sc), one rounding.  The limb
// sum is rounded to odd in fp64 and then to fp32: a value rounded to odd with
// 53 >= 24 + 2 bits rounds to nearest exactly as the exact value does, in the
// normal and subnormal fp32 ranges alike, as long as the scaling by 2^sc is
// exact in fp64 (true unless the fp64 value is subnormal, which rounds the
// multiword integer to 24 bits directly).
template <int T>
O2M_HD inline float lift_round_f32(const double (&S)[T], const double *mlimb, double inv_m, int sc) {
    double c[T];
    lift_limbs<T>(S, mlimb, inv_m, c);
    double x;
    if constexpr (T == 2) {
        x = sum_round_odd(c[1] * kTwo40, c[0]);
    } else if constexpr (T == 3) {
        x = sum3_ro(c[2] * kTwo80, c[1] * kTwo40, c[0]);
    } else {
        double a, b, low;
        top3_of<T>(c, a, b, low);
        x = sum3_ro(a, b, low);
    }
    const double r = ldexp(x, sc);
    if (x == 0.0 || !(fabs(r) < 0x1p-1022)) return (float)r;
    return (float)round_words_fmt<LimbWords<T>::value, 24, -126>(words_of<T>(c), sc);
}

// The lifted limbs rounded once (tests): the same steps as lift_round /
// lift_round_f32 after lift_limbs.
template <int T>
O2M_HD inline double round_lifted(const double (&c_in)[T], int sc, bool f32) {
    // S = c with q = 0: lift_limbs leaves the limbs as they are when M's
    // limbs are zero and 1/M is zero
    const double zero[T] = {};
    return f32 ? (double)lift_round_f32<T>(c_in, zero, 0.0, sc) : lift_round<T>(c_in, zero, 0.0, sc);
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
