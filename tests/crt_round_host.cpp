// Host build of the CRT rounding helpers, for tests/test_crt_round.py.
#define O2M_HD
#include "../paper_2609_05419_amd/csrc/crt_round.h"

namespace {
template <int T>
double lift(const double *S, const double *mlimb, double inv_m, int sc, int f32) {
    double s[T];
    for (int t = 0; t < T; ++t) s[t] = S[t];
    return f32 ? (double)o2m::lift_round_f32<T>(s, mlimb, inv_m, sc) : o2m::lift_round<T>(s, mlimb, inv_m, sc);
}

template <int W>
double round_fmt(const int64_t *limbs, int T, int sc, int f32) {
    o2m::UW<W> v = {};
    for (int t = 0; t < T; ++t) o2m::add_shifted<W>(v, limbs[t], 40 * t);
    return f32 ? o2m::round_words_fmt<W, 24, -126>(v, sc) : o2m::round_words_fmt<W, 53, -1022>(v, sc);
}
}  // namespace

extern "C" {
double t_sum3_rn(double a, double b, double c) { return o2m::sum3_rn(a, b, c); }
double t_round3_rn(double c0, double c1, double c2) { return o2m::round3_rn(c0, c1, c2); }
double t_sum3_ro(double a, double b, double c) { return o2m::sum3_ro(a, b, c); }
double t_sum_ro(double a, double b) { return o2m::sum_round_odd(a, b); }
// T limbs (T <= 6) rounded into fp64 (f32 = 0) or fp32 (f32 = 1) after 2^sc
double t_round_limbs_fmt(const int64_t *limbs, int T, int sc, int f32) {
    return T <= 4 ? round_fmt<3>(limbs, T, sc, f32) : round_fmt<4>(limbs, T, sc, f32);
}
double t_round_limbs(const int64_t *limbs, int T, int sc) {
    if (T <= 4) {
        o2m::UW<3> v = {};
        for (int t = 0; t < T; ++t) o2m::add_shifted<3>(v, limbs[t], 40 * t);
        return o2m::round_words<3>(v, sc);
    }
    o2m::UW<4> v = {};
    for (int t = 0; t < T; ++t) o2m::add_shifted<4>(v, limbs[t], 40 * t);
    return o2m::round_words<4>(v, sc);
}
// lifted limbs (|c_t| < 2^53) rounded once into fp64 / fp32 after 2^sc
double t_round_lifted(const double *c, int T, int sc, int f32) {
    double c2[2], c3[3], c4[4], c5[5], c6[6];
    switch (T) {
    case 2: for (int t = 0; t < 2; ++t) c2[t] = c[t]; return o2m::round_lifted<2>(c2, sc, f32 != 0);
    case 3: for (int t = 0; t < 3; ++t) c3[t] = c[t]; return o2m::round_lifted<3>(c3, sc, f32 != 0);
    case 4: for (int t = 0; t < 4; ++t) c4[t] = c[t]; return o2m::round_lifted<4>(c4, sc, f32 != 0);
    case 5: for (int t = 0; t < 5; ++t) c5[t] = c[t]; return o2m::round_lifted<5>(c5, sc, f32 != 0);
    default: for (int t = 0; t < 6; ++t) c6[t] = c[t]; return o2m::round_lifted<6>(c6, sc, f32 != 0);
    }
}
double t_lift_round(const double *S, int T, const double *mlimb, double inv_m, int sc, int f32) {
    switch (T) {
    case 2: return lift<2>(S, mlimb, inv_m, sc, f32);
    case 3: return lift<3>(S, mlimb, inv_m, sc, f32);
    case 4: return lift<4>(S, mlimb, inv_m, sc, f32);
    case 5: return lift<5>(S, mlimb, inv_m, sc, f32);
    default: return lift<6>(S, mlimb, inv_m, sc, f32);
    }
}
}
