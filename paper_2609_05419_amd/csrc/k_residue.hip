// K2: quantization, residues and the 2M pre step (Algorithm 1 steps 3-4,
// eq. 2m-pre).
//
// For every entry x = a 2^(p - E_r) of an operand (componentwise, rounded to
// the nearest integer, ties to even: step 3) and every 2M modulus m_l with
// root s_l, the kernel writes the two int8 residues
//     A+ = (x_re + s x_im) mod m,   A- = (x_re - s x_im) mod m      (eq. 2m-pre)
// in the symmetric range [-(m-1)/2, (m-1)/2] into the operand planes 2l and
// 2l+1, in the fragment order the int8 GEMM consumes (o2m_internal.h).  For
// the 3M moduli of a hybrid set it writes x_re, x_im and x_re + x_im mod m
// into three planes (3M after reduction, Section 3.2); for even m = 256 the
// low byte of the residue in [-128, 128] is the int8 residue (-128 = 128).
//
// Exact residues without integer division: x (an integer held exactly in a
// double) is split into D base-2^26 digits x = sum_d x_d 2^(26 d), peeled
// from the top so that |x_d| <= 2^25 below the top digit; then
// R = sum_d c_d x_d = x (mod m) with c_d = 2^(26 d) mod m (symmetric),
// likewise I for x_im.  The host picks D from the bound on |x| so that the top
// digit stays below 2^36 (D = 2 up to 2^62, 3 up to 2^88; D = 4, 5 keep it
// below 2^30 and hold the digits as int32), which keeps |R| < 2^43.01 and
// A+- = R +- s I an exact integer below 2^51 (s <= 120).  Up to |x| <= 2^44
// no split is needed (D = 1: R = x, and |A+-| <= 121 2^44 < 2^51).  q = rint(A / m)
// comes out of one fma against 1.5 2^52 (the low word of the sum is q), and
// A - q m, needed only modulo 2^8, is one 24-bit integer multiply-add on the
// low words.
//
// Bound: HBM.  Algorithmic bytes per complex fp64 input element:
// 16 read + 2N written (8 + 2N for fp32 input).
#include "o2m_internal.h"

#include <type_traits>

namespace o2m {
namespace {

constexpr double kMagic = 6755399441055744.0;  // 1.5 * 2^52

// Digit storage: exact doubles for D <= 3, int32 for D >= 4 (digits < 2^30).
template <int D> struct Digit { typedef double type; };
template <> struct Digit<4> { typedef int type; };
template <> struct Digit<5> { typedef int type; };

// x = sum_d dg[d] 2^(26 d), peeled from the top digit down (each step exact).
template <int D, int PT, typename DT>
__device__ inline void split_digits(double x, DT (&dg)[D][PT], int e) {
#pragma unroll
    for (int d = D - 1; d >= 1; --d) {
        const double q = rint(ldexp(x, -26 * d));
        x = fma(-q, ldexp(1.0, 26 * d), x);
        dg[d][e] = (DT)q;
    }
    dg[0][e] = (DT)x;
}

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

// k entries per thread: one lane chunk of a fragment (16), or half of one for
// four and five digits, whose int32 digits would otherwise hold the kernel to
// one wave per SIMD; a fragment then goes to two waves, 32 chunks each.
template <int D> constexpr int per_thread() { return D >= 4 ? 8 : 16; }

// PT residue bytes of one lane, contiguous in the plane (16- or 8-byte store).
// The stores are non-temporal (no cache allocation): the planes are far
// larger than the caches and are read back only by the GEMM, from its own
// tile windows; plain stores measured 4-5% slower for the whole pass.
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
template <int PT>
__device__ inline void store_words(int8_t *dst, const uint32_t (&w)[PT / 4]) {
    if constexpr (PT == 16) {
        const u32x4 v = {w[0], w[1], w[2], w[3]};
        __builtin_nontemporal_store(v, reinterpret_cast<u32x4 *>(dst));
    } else {
        const u32x2 v = {w[0], w[1]};
        __builtin_nontemporal_store(v, reinterpret_cast<u32x2 *>(dst));
    }
}

// MODE 0: rows of X (A, column-major m x k): entry (r, kk) at X[r + kk*ld]
// MODE 1: columns of X (B, column-major k x n): entry (r, kk) at X[kk + r*ld]
// MODE 2: SYRK, X real column-major n x k: (r, kk) = X[r + kk ld] + i X[r + (kk+kh) ld]
// conj: the operand is the complex conjugate of X (imaginary parts negated)
// D: base-2^26 digits of the quantized values (1..5, from their bound)
// PAIRS (complex fp32, the host sets it when every pair is 16-byte aligned):
// MODE 1 reads two consecutive entries of a column of B per 16-byte load;
// MODE 0 reads rows 2i, 2i + 1 of a column of A per 16-byte load, the even
// lane of a lane pair columns kk0..kk0+7 and the odd lane kk0+8..kk0+15, and
// the pair then swaps halves so that each lane holds its own row's 16 entries
template <int MODE, ElemType ET, int D, bool SCALED, bool PAIRS = false>
__global__ __launch_bounds__(256, D == 1 ? 3 : 1) void residue_kernel(const void *X, int ld, const int32_t *E,
                                                      int shift, int khalf, int kreal, int rows, int k,
                                                      int rows_pad, int kblocks, int plane_kblocks,
                                                      int kofs_p, int kofs_m, size_t plane_bytes,
                                                      int conj, ResidueParams rp, int8_t *planes) {
    constexpr int PT = per_thread<D>();
    constexpr int kHalves = 16 / PT;                          // waves per fragment
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(blockIdx.x * 4 + (threadIdx.x >> 6));  // wave-uniform
    const int frag = wave / kHalves, half = wave % kHalves;   // one fragment per kHalves waves
    const int frows = rows_pad / kFragRows;                   // fragments along rows
    const int fks = kblocks;                                  // fragments along k
    int fr, fk;
    if (frag >= frows * fks) return;
    if (MODE == 1) { fk = frag % fks; fr = frag / fks; }      // B: walk k fastest (contiguous)
    else { fr = frag % frows; fk = frag / frows; }            // A: walk rows fastest
    // the fragment's 16-byte lane chunk and the part of it this lane fills;
    // with two waves per fragment each takes 32 whole chunks (adjacent lanes
    // fill the two halves of one), so that a store covers 512 contiguous bytes
    const int chunk = kHalves == 1 ? lane : half * 32 + (lane >> 1);
    const int part = kHalves == 1 ? 0 : lane & 1;
    const int r = fr * kFragRows + (chunk & 15);
    const int kk0 = fk * kStageK + (chunk >> 4) * 16 + part * PT;

    // ---- load and quantize (step 3) -------------------------------------
    // A wave whose fragment (16 rows x 64 k) lies inside the operand takes
    // every load unguarded, so all of them are in flight before the first is
    // used; the guarded form is taken at the edges only.  (With a per-lane
    // guard around each load the compiler moves the quantization of the value
    // into the guarded branch, where it must wait for that load: the loads
    // then went out one at a time.)
    typedef typename Digit<D>::type DT;
    DT xr[D][PT], xi[D][PT];
    const bool inner = fr * kFragRows + kFragRows <= rows && fk * kStageK + kStageK <= k &&
                       (MODE != 2 || fk * kStageK + kStageK + khalf <= kreal);
    // the row's exponent is fetched first and used once the entries' loads
    // are issued (every padded row has an entry)
    int erow = 0;
    if constexpr (SCALED) erow = E[r];
    int sh = 0;
    bool live = r < rows;                    // bounds only until settle()
    auto settle = [&]() {
        if constexpr (SCALED) {
            live = live && erow != INT32_MIN;  // non-finite row: output masked later
            sh = shift - erow;
        }
    };
    auto put = [&](int e, double vr, double vi) {
        if (!live) vr = vi = 0.0;
        if (conj) vi = -vi;                  // conjugated operand: exact
        if (SCALED) {
            vr = rint(ldexp(vr, sh));
            vi = rint(ldexp(vi, sh));
        }
        split_digits<D, PT>(vr, xr, e);
        split_digits<D, PT>(vi, xi, e);
    };
    auto load_all = [&](auto edge) {
        constexpr bool EDGE = decltype(edge)::value;
        if constexpr (PAIRS && MODE == 0) {
            static_assert(ET == kF32 && PT == 16, "pairs of complex fp32 rows, one lane chunk per lane");
            const bool odd = lane & 1;
            const int re = r - (int)odd;                 // the pair's even row
            const float2 *Xa = reinterpret_cast<const float2 *>(X);
            float4 v[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const int kk = kk0 + (odd ? 8 : 0) + j;
                v[j] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
                if (!EDGE) {
                    v[j] = *reinterpret_cast<const float4 *>(Xa + (size_t)re + (size_t)kk * ld);
                } else if (kk < k) {
                    if (re + 1 < rows) {
                        v[j] = *reinterpret_cast<const float4 *>(Xa + (size_t)re + (size_t)kk * ld);
                    } else if (re < rows) {
                        const float2 t = Xa[(size_t)re + (size_t)kk * ld];
                        v[j].x = t.x;
                        v[j].y = t.y;
                    }
                }
            }
            settle();
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                // the even lane passes on its odd row's half, the odd lane its even row's
                const float rx = __shfl_xor(odd ? v[j].x : v[j].z, 1, 64);
                const float ry = __shfl_xor(odd ? v[j].y : v[j].w, 1, 64);
                put(j, odd ? rx : v[j].x, odd ? ry : v[j].y);
                put(8 + j, odd ? v[j].z : rx, odd ? v[j].w : ry);
            }
        } else if constexpr (PAIRS) {
            static_assert(MODE == 1 && ET == kF32, "pairs of complex fp32 entries along a column");
            const float2 *Xc = reinterpret_cast<const float2 *>(X) + (size_t)r * ld;
            float4 v[PT / 2];
#pragma unroll
            for (int e = 0; e < PT; e += 2) {
                const int kk = kk0 + e;
                v[e / 2] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
                if (!EDGE) {
                    v[e / 2] = *reinterpret_cast<const float4 *>(Xc + kk);
                } else if (live && kk + 1 < k) {
                    v[e / 2] = *reinterpret_cast<const float4 *>(Xc + kk);
                } else if (live && kk < k) {
                    const float2 t = Xc[kk];
                    v[e / 2].x = t.x;
                    v[e / 2].y = t.y;
                }
            }
            settle();
#pragma unroll
            for (int e = 0; e < PT; e += 2) {
                put(e, (double)v[e / 2].x, (double)v[e / 2].y);
                put(e + 1, (double)v[e / 2].z, (double)v[e / 2].w);
            }
        } else {
            double vr[PT], vi[PT];
#pragma unroll
            for (int e = 0; e < PT; ++e) {
                const int kk = kk0 + e;
                vr[e] = 0.0;
                vi[e] = 0.0;
                if (!EDGE || (live && kk < k)) {
                    if (MODE == 0) {
                        const double2 v = Load<ET>::get(X, (size_t)r + (size_t)kk * ld);
                        vr[e] = v.x; vi[e] = v.y;
                    } else if (MODE == 1) {
                        const double2 v = Load<ET>::get(X, (size_t)kk + (size_t)r * ld);
                        vr[e] = v.x; vi[e] = v.y;
                    } else {
                        const double *Xr = reinterpret_cast<const double *>(X);
                        vr[e] = Xr[(size_t)r + (size_t)kk * ld];
                        if (!EDGE || kk + khalf < kreal) vi[e] = Xr[(size_t)r + (size_t)(kk + khalf) * ld];
                    }
                }
            }
            settle();
#pragma unroll
            for (int e = 0; e < PT; ++e) put(e, vr[e], vi[e]);
        }
    };
    if (__builtin_expect(inner, 1)) load_all(std::false_type());
    else load_all(std::true_type());

    // ---- residues and 2M pre per modulus (step 4, eq. 2m-pre) -------------
    int8_t *dst_p = planes + plane_offset(r, kk0 + kofs_p * kStageK, plane_kblocks);
    int8_t *dst_m = planes + plane_offset(r, kk0 + kofs_m * kStageK, plane_kblocks) + plane_bytes;
    for (int l = 0; l < rp.n2; ++l) {
        const double inv = rp.inv[l];
        const double s = (double)rp.root[l];
        const uint32_t negm = (uint32_t)(-rp.mod[l]) & 0xFFFFFFu;
        uint32_t wp[PT / 4], wm[PT / 4];
#pragma unroll
        for (int q = 0; q < PT / 4; ++q) {
            uint32_t bp[4], bm[4];
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                const int e = 4 * q + t;
                double R = (double)xr[0][e], I = (double)xi[0][e];
#pragma unroll
                for (int d = 1; d < D; ++d) {
                    R = fma(rp.cpow[l][d - 1], (double)xr[d][e], R);
                    I = fma(rp.cpow[l][d - 1], (double)xi[d][e], I);
                }
                const double Ap = fma(s, I, R), Am = fma(-s, I, R);
                const double tp = fma(Ap, inv, kMagic), tm = fma(Am, inv, kMagic);
                const uint32_t ap = lo32(Ap + kMagic), am = lo32(Am + kMagic);
                bp[t] = mad24(lo32(tp), negm, ap);   // A+ - q m (low byte)
                bm[t] = mad24(lo32(tm), negm, am);
            }
            wp[q] = pack4(bp[0], bp[1], bp[2], bp[3]);
            wm[q] = pack4(bm[0], bm[1], bm[2], bm[3]);
        }
        store_words<PT>(dst_p + (size_t)(2 * l) * plane_bytes, wp);
        store_words<PT>(dst_m + (size_t)(2 * l) * plane_bytes, wm);
    }

    // ---- hybrid sets: residues of Xr, Xi and Xr + Xi for 3M (Section 3.2) ---
    for (int l = rp.n2; l < rp.n; ++l) {
        const double inv = rp.inv[l];
        const uint32_t negm = (uint32_t)(-rp.mod[l]) & 0xFFFFFFu;
        uint32_t w[3][PT / 4];
#pragma unroll
        for (int q = 0; q < PT / 4; ++q) {
            uint32_t by[3][4];
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                const int e = 4 * q + t;
                double R = (double)xr[0][e], I = (double)xi[0][e];
#pragma unroll
                for (int d = 1; d < D; ++d) {
                    R = fma(rp.cpow[l][d - 1], (double)xr[d][e], R);
                    I = fma(rp.cpow[l][d - 1], (double)xi[d][e], I);
                }
                const double v[3] = {R, I, R + I};
#pragma unroll
                for (int c = 0; c < 3; ++c) {
                    const double tq = fma(v[c], inv, kMagic);
                    by[c][t] = mad24(lo32(tq), negm, lo32(v[c] + kMagic));
                }
            }
#pragma unroll
            for (int c = 0; c < 3; ++c) w[c][q] = pack4(by[c][0], by[c][1], by[c][2], by[c][3]);
        }
        const size_t p0 = (size_t)(2 * rp.n2 + 3 * (l - rp.n2));
#pragma unroll
        for (int c = 0; c < 3; ++c)
            store_words<PT>(dst_p + (p0 + c) * plane_bytes, w[c]);
    }
}

}  // namespace

hipError_t launch_residues(int mode, ElemType et, const void *X, int ld, const int32_t *E, int shift,
                           int digits, int khalf, const PlaneGeom &g, const ResidueParams &rp,
                           int8_t *planes, hipStream_t st) {
    const int kreal = khalf > 0 ? g.kreal : 0;
    // waves: one per fragment, two for four and five digits (per_thread)
    const long frags = (long)(g.rows_pad / kFragRows) * (long)g.kblocks;
    const long waves = frags * (digits >= 4 ? 2 : 1);
    if ((waves + 3) / 4 > 0x7FFFFFFF) return hipErrorInvalidValue;
    const unsigned blocks = (unsigned)((waves + 3) / 4);
    // complex fp32 entries in 16-byte pairs when every pair is aligned: along
    // a column of B (k-chunks start at even k) or across rows 2i, 2i + 1 of A
    // (lane chunks of one row, up to three digits); an even ld and a 16-byte
    // aligned base suffice
    const bool pairs = et == kF32 && (mode == 1 || digits <= 3) && ld % 2 == 0 && ((uintptr_t)X & 15) == 0;
#define O2M_RES(M, T, DD, SC, PR)                                                                \
    residue_kernel<M, T, DD, SC, PR><<<blocks, 256, 0, st>>>(X, ld, E, shift, khalf, kreal, g.rows, g.k, \
                                                            g.rows_pad, g.kblocks, g.plane_kblocks, \
                                                            g.kofs_p, g.kofs_m, g.plane_bytes, g.conj, rp, \
                                                            planes)
#define O2M_RES_D(M, T, PR)                                   \
    switch (digits) {                                         \
    case 1: O2M_RES(M, T, 1, true, PR); break;                \
    case 2: O2M_RES(M, T, 2, true, PR); break;                \
    case 3: O2M_RES(M, T, 3, true, PR); break;                \
    case 4: O2M_RES(M, T, 4, true, PR); break;                \
    case 5: O2M_RES(M, T, 5, true, PR); break;                \
    default: return hipErrorInvalidValue;                     \
    }
    if (mode == 0 && et == kF64) { O2M_RES_D(0, kF64, false) }
    else if (mode == 1 && et == kF64) { O2M_RES_D(1, kF64, false) }
    else if (mode == 0 && et == kF32 && pairs) {
        switch (digits) {
        case 1: O2M_RES(0, kF32, 1, true, true); break;
        case 2: O2M_RES(0, kF32, 2, true, true); break;
        case 3: O2M_RES(0, kF32, 3, true, true); break;
        default: return hipErrorInvalidValue;
        }
    }
    else if (mode == 0 && et == kF32) { O2M_RES_D(0, kF32, false) }
    else if (mode == 1 && et == kF32 && pairs) { O2M_RES_D(1, kF32, true) }
    else if (mode == 1 && et == kF32) { O2M_RES_D(1, kF32, false) }
    else if (mode == 2 && et == kR64) { O2M_RES_D(2, kR64, false) }
    else if (mode == 0 && et == kI32) O2M_RES(0, kI32, 2, false, false);
    else if (mode == 1 && et == kI32) O2M_RES(1, kI32, 2, false, false);
    else return hipErrorInvalidValue;
#undef O2M_RES_D
#undef O2M_RES
    return hipGetLastError();
}

}  // namespace o2m
