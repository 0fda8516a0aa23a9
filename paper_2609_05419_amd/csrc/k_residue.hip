// K2: quantization, residues and the 2M pre step (Algorithm 1 steps 3-4,
// eq. 2m-pre).
//
// For every entry x = a 2^(p - E_r) of an operand (componentwise, rounded to
// the nearest integer, ties to even: step 3) and every 2M modulus m_l with
// root s_l, the kernel writes the two int8 residues
//     A+ = (x_re + s x_im) mod m,   A- = (x_re - s x_im) mod m      (eq. 2m-pre)
// in the symmetric range [-(m-1)/2, (m-1)/2] into the operand planes 2l and
// 2l+1, in the fragment order the int8 GEMM consumes (o2m_internal.h).
//
// Exact residues without integer division: x (an integer held exactly in a
// double, |x| <= 2^pA) is split as x = x2 2^52 + x1 2^26 + x0 with
// |x1|, |x0| <= 2^25; then R = c52 x2 + c26 x1 + x0 = x (mod m) with
// c = 2^26, 2^52 mod m (symmetric), likewise I for x_im, and A+- = R +- s I is
// an exact integer below 2^52.  q = rint(A / m) comes out of one fma against
// 1.5 2^52 (the low word of the sum is q), and A - q m, needed only modulo
// 2^8, is one 24-bit integer multiply-add on the low words.
//
// Bound: HBM.  Algorithmic bytes per complex fp64 input element:
// 16 read + 2N written (8 + 2N for fp32 input).
#include "o2m_internal.h"

namespace o2m {
namespace {

constexpr double kMagic = 6755399441055744.0;  // 1.5 * 2^52
constexpr double kTwo26 = 67108864.0;
constexpr double kTwoM26 = 1.0 / 67108864.0;
constexpr double kTwo52 = 4503599627370496.0;
constexpr double kTwoM52 = 1.0 / 4503599627370496.0;

template <ElemType ET> struct Load;
template <> struct Load<kF64> {
    static __device__ inline double2 get(const void *X, size_t idx) {
        return reinterpret_cast<const double2 *>(X)[idx];
    }
};
template <> struct Load<kF32> {
    static __device__ inline double2 get(const void *X, size_t idx) {
        const float2 v = reinterpret_cast<const float2 *>(X)[idx];
        return make_double2((double)v.x, (double)v.y);
    }
};
template <> struct Load<kR64> {
    static __device__ inline double2 get(const void *X, size_t idx) {
        return make_double2(reinterpret_cast<const double *>(X)[idx], 0.0);
    }
};
template <> struct Load<kI32> {
    static __device__ inline double2 get(const void *X, size_t idx) {
        const int2 v = reinterpret_cast<const int2 *>(X)[idx];
        return make_double2((double)v.x, (double)v.y);
    }
};

__device__ inline uint32_t lo32(double d) { return (uint32_t)__double2loint(d); }

// a * b + c on the low 24 bits of a and b (v_mad_u32_u24)
__device__ inline uint32_t mad24(uint32_t a, uint32_t b, uint32_t c) { return __umul24(a, b) + c; }

__device__ inline uint32_t pack4(uint32_t b0, uint32_t b1, uint32_t b2, uint32_t b3) {
    const uint32_t lo = __builtin_amdgcn_perm(b1, b0, 0x0c0c0400u);  // [b0.0, b1.0, 0, 0]
    const uint32_t hi = __builtin_amdgcn_perm(b3, b2, 0x0c0c0400u);
    return __builtin_amdgcn_perm(hi, lo, 0x05040100u);                // [lo.0, lo.1, hi.0, hi.1]
}

constexpr int kPerThread = 16;  // k entries per thread = one lane chunk of a fragment

// MODE 0: rows of X (A, column-major m x k): entry (r, kk) at X[r + kk*ld]
// MODE 1: columns of X (B, column-major k x n): entry (r, kk) at X[kk + r*ld]
// MODE 2: SYRK, X real column-major n x k: (r, kk) = X[r + kk ld] + i X[r + (kk+kh) ld]
// SPLIT3: quantized values may exceed 2^62 (three-way split needed)
template <int MODE, ElemType ET, bool SPLIT3, bool SCALED>
__global__ __launch_bounds__(256) void residue_kernel(const void *X, int ld, const int32_t *E,
                                                      int shift, int khalf, int kreal, int rows, int k,
                                                      int rows_pad, int kblocks, int plane_kblocks,
                                                      int kofs_p, int kofs_m, size_t plane_bytes,
                                                      ResidueParams rp, int8_t *planes) {
    const int lane = threadIdx.x & 63;
    const int wave = blockIdx.x * 4 + (threadIdx.x >> 6);   // one wave = one fragment
    const int frows = rows_pad / kFragRows;                   // fragments along rows
    const int fks = kblocks;                                  // fragments along k
    int fr, fk;
    if (wave >= frows * fks) return;
    if (MODE == 1) { fk = wave % fks; fr = wave / fks; }      // B: walk k fastest (contiguous)
    else { fr = wave % frows; fk = wave / frows; }            // A: walk rows fastest
    const int r = fr * kFragRows + (lane & 15);
    const int kk0 = fk * kStageK + (lane >> 4) * 16;

    // ---- load and quantize (step 3) -------------------------------------
    double x1r[kPerThread], x0r[kPerThread], x1i[kPerThread], x0i[kPerThread];
    double x2r[SPLIT3 ? kPerThread : 1], x2i[SPLIT3 ? kPerThread : 1];
    int sh = 0;
    bool live = r < rows;
    if (SCALED && live) {
        const int e = E[r];
        if (e == INT32_MIN) live = false;    // non-finite row: output masked later
        else sh = shift - e;
    }
#pragma unroll
    for (int e = 0; e < kPerThread; ++e) {
        const int kk = kk0 + e;
        double vr = 0.0, vi = 0.0;
        if (live && kk < k) {
            if (MODE == 0) {
                const double2 v = Load<ET>::get(X, (size_t)r + (size_t)kk * ld);
                vr = v.x; vi = v.y;
            } else if (MODE == 1) {
                const double2 v = Load<ET>::get(X, (size_t)kk + (size_t)r * ld);
                vr = v.x; vi = v.y;
            } else {
                const double *Xr = reinterpret_cast<const double *>(X);
                vr = Xr[(size_t)r + (size_t)kk * ld];
                if (kk + khalf < kreal) vi = Xr[(size_t)r + (size_t)(kk + khalf) * ld];
            }
        }
        if (SCALED) {
            vr = rint(ldexp(vr, sh));
            vi = rint(ldexp(vi, sh));
        }
        if (SPLIT3) {
            x2r[e] = rint(vr * kTwoM52); vr = fma(-x2r[e], kTwo52, vr);
            x2i[e] = rint(vi * kTwoM52); vi = fma(-x2i[e], kTwo52, vi);
        }
        x1r[e] = rint(vr * kTwoM26); x0r[e] = fma(-x1r[e], kTwo26, vr);
        x1i[e] = rint(vi * kTwoM26); x0i[e] = fma(-x1i[e], kTwo26, vi);
    }

    // ---- residues and 2M pre per modulus (step 4, eq. 2m-pre) -------------
    int8_t *dst_p = planes + plane_offset(r, kk0 + kofs_p * kStageK, plane_kblocks);
    int8_t *dst_m = planes + plane_offset(r, kk0 + kofs_m * kStageK, plane_kblocks) + plane_bytes;
    for (int l = 0; l < rp.n; ++l) {
        const double c26 = rp.c26[l], c52 = rp.c52[l], inv = rp.inv[l];
        const double s = (double)rp.root[l];
        const uint32_t negm = (uint32_t)(-rp.mod[l]) & 0xFFFFFFu;
        uint32_t wp[4], wm[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            uint32_t bp[4], bm[4];
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                const int e = 4 * q + t;
                double R = fma(c26, x1r[e], x0r[e]);
                double I = fma(c26, x1i[e], x0i[e]);
                if (SPLIT3) { R = fma(c52, x2r[e], R); I = fma(c52, x2i[e], I); }
                const double Ap = fma(s, I, R), Am = fma(-s, I, R);
                const double tp = fma(Ap, inv, kMagic), tm = fma(Am, inv, kMagic);
                const uint32_t ap = lo32(Ap + kMagic), am = lo32(Am + kMagic);
                bp[t] = mad24(lo32(tp), negm, ap);   // A+ - q m (low byte)
                bm[t] = mad24(lo32(tm), negm, am);
            }
            wp[q] = pack4(bp[0], bp[1], bp[2], bp[3]);
            wm[q] = pack4(bm[0], bm[1], bm[2], bm[3]);
        }
        *reinterpret_cast<uint4 *>(dst_p + (size_t)(2 * l) * plane_bytes) = make_uint4(wp[0], wp[1], wp[2], wp[3]);
        *reinterpret_cast<uint4 *>(dst_m + (size_t)(2 * l) * plane_bytes) = make_uint4(wm[0], wm[1], wm[2], wm[3]);
    }
}

}  // namespace

hipError_t launch_residues(int mode, ElemType et, const void *X, int ld, const int32_t *E, int shift,
                           bool wide, int khalf, const PlaneGeom &g, const ResidueParams &rp,
                           int8_t *planes, hipStream_t st) {
    const int kreal = khalf > 0 ? g.kreal : 0;
    const long waves = (long)(g.rows_pad / kFragRows) * (long)g.kblocks;
    const unsigned blocks = (unsigned)((waves + 3) / 4);
    const bool split3 = wide;
#define O2M_RES(M, T, S3, SC)                                                                    \
    residue_kernel<M, T, S3, SC><<<blocks, 256, 0, st>>>(X, ld, E, shift, khalf, kreal, g.rows, g.k,     \
                                                        g.rows_pad, g.kblocks, g.plane_kblocks,   \
                                                        g.kofs_p, g.kofs_m, g.plane_bytes, rp,    \
                                                        planes)
    if (mode == 0 && et == kF64) { if (split3) O2M_RES(0, kF64, true, true); else O2M_RES(0, kF64, false, true); }
    else if (mode == 1 && et == kF64) { if (split3) O2M_RES(1, kF64, true, true); else O2M_RES(1, kF64, false, true); }
    else if (mode == 0 && et == kF32) { if (split3) O2M_RES(0, kF32, true, true); else O2M_RES(0, kF32, false, true); }
    else if (mode == 1 && et == kF32) { if (split3) O2M_RES(1, kF32, true, true); else O2M_RES(1, kF32, false, true); }
    else if (mode == 2 && et == kR64) { if (split3) O2M_RES(2, kR64, true, true); else O2M_RES(2, kR64, false, true); }
    else if (mode == 0 && et == kI32) O2M_RES(0, kI32, false, false);
    else if (mode == 1 && et == kI32) O2M_RES(1, kI32, false, false);
    else return hipErrorInvalidValue;
#undef O2M_RES
    return hipGetLastError();
}

}  // namespace o2m
