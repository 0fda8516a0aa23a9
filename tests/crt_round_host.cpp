// Host build of the CRT rounding helpers, for tests/test_crt_round.py.
#define O2M_HD
#include "../paper_2609_05419_amd/csrc/crt_round.h"

extern "C" {
double t_sum3_rn(double a, double b, double c) { return o2m::sum3_rn(a, b, c); }
double t_round_limbs(const int64_t *limbs, int T, int sc) {
    o2m::U192 v = {0, 0, 0};
    for (int t = 0; t < T; ++t) o2m::add_shifted(v, limbs[t], 40 * t);
    return o2m::round_u192(v, sc);
}
double t_lift_round(const double *S, int T, const double *mlimb, double inv_m, int sc) {
    if (T == 2) { const double s[2] = {S[0], S[1]}; return o2m::lift_round<2>(s, mlimb, inv_m, sc); }
    if (T == 3) { const double s[3] = {S[0], S[1], S[2]}; return o2m::lift_round<3>(s, mlimb, inv_m, sc); }
    const double s[4] = {S[0], S[1], S[2], S[3]};
    return o2m::lift_round<4>(s, mlimb, inv_m, sc);
}
}
