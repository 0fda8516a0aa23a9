// K4: 2M post step, CRT, symmetric lift and inverse scaling (eq. 2m-post and
// Algorithm 1 steps 5-7).
//
// Per output entry and modulus m_l the int8 GEMM left r+ = C+ mod m and
// r- = C- mod m (symmetric).  The 2M post step gives
//     Re c = 2^-1 (r- + r+),  Im c = s 2^-1 (r- - r+)   (mod m)     (eq. 2m-post)
// and since the CRT is linear modulo M, the constants 2^-1 and s 2^-1 are
// folded into the CRT weights: with u = r- + r+ and v = r- - r+,
//     X_re = sum_l u_l W^re_l = Re c (mod M),   X_im = sum_l v_l W^im_l.
// The weights are held as T balanced base-2^40 limbs, so every limb sum
// S_t = sum_l u_l w_lt is an exact fp64 integer (|S_t| < 2^52).  The quotient
// q = rint(X / M) is estimated from a fp64 Horner sum; the scaling budget keeps
// |c| / M <= 1/2 - 2^-32, far from the rounding boundary, so q is exact.  The
// lifted value c = X - q M (step 6) is then exact as limbs c_t = S_t - q M_t,
// assembled into a 192-bit two's complement integer and rounded to the nearest
// double, ties to even, and scaled by 2^(E_i + F_j - pA - pB) (step 7).
//
// Bound: HBM.  Algorithmic bytes per output entry: 2N residues read + 16
// written (complex fp64; 8 for complex fp32).
#include "o2m_internal.h"

namespace o2m {
namespace {

constexpr double kTwo40 = 1099511627776.0;

struct U192 {
    uint64_t w0, w1, w2;
};

// a += x * 2^s (two's complement, modulo 2^192); s is a compile-time multiple of 40
__device__ inline void add_shifted(U192 &a, int64_t x, int s) {
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

// Round the 192-bit signed integer v to the nearest double (ties to even) and
// multiply by 2^sc, rounding once.
__device__ inline double round_scaled(U192 v, int sc) {
    const bool neg = (int64_t)v.w2 < 0;
    if (neg) {
        v.w0 = ~v.w0; v.w1 = ~v.w1; v.w2 = ~v.w2;
        v.w0 += 1;
        const uint64_t c0 = v.w0 == 0;
        v.w1 += c0;
        v.w2 += (c0 && v.w1 == 0);
    }
    int lz;
    if (v.w2) lz = __clzll(v.w2);
    else if (v.w1) lz = 64 + __clzll(v.w1);
    else if (v.w0) lz = 128 + __clzll(v.w0);
    else return 0.0;
    uint64_t h, rest_nonzero;
    if (lz >= 128) {
        h = v.w0 << (lz - 128);
        rest_nonzero = 0;
    } else if (lz >= 64) {
        const int s = lz - 64;
        h = s ? (v.w1 << s) | (v.w0 >> (64 - s)) : v.w1;
        rest_nonzero = s ? (v.w0 << s) : v.w0;
    } else {
        const int s = lz;
        h = s ? (v.w2 << s) | (v.w1 >> (64 - s)) : v.w2;
        const uint64_t n1 = s ? (v.w1 << s) | (v.w0 >> (64 - s)) : v.w1;
        const uint64_t n0 = s ? (v.w0 << s) : v.w0;
        rest_nonzero = n1 | n0;
    }
    uint64_t mant = h >> 11;
    const uint64_t rb = h & 0x7FF;
    if (rb > 0x400 || (rb == 0x400 && (rest_nonzero != 0 || (mant & 1)))) mant += 1;
    const int top = 191 - lz;
    const double r = ldexp((double)mant, top - 52 + sc);
    return neg ? -r : r;
}

// Step 5-6: from the limb sums, the exact lifted integer c as 192 bits.
template <int T>
__device__ inline U192 lift(const double (&S)[T], const CrtParams &cp) {
    double X = S[T - 1];
#pragma unroll
    for (int t = T - 2; t >= 0; --t) X = fma(X, kTwo40, S[t]);
    const double q = rint(X * cp.inv_m);
    U192 v = {0, 0, 0};
#pragma unroll
    for (int t = 0; t < T; ++t) {
        const double ct = fma(-q, cp.mlimb[t], S[t]);
        add_shifted(v, (int64_t)ct, 40 * t);
    }
    return v;
}

__device__ inline int sext8(uint32_t w, int e) { return (int)(int8_t)(w >> (8 * e)); }

template <ElemType OT> struct Out;
template <> struct Out<kF64> {
    static __device__ inline void put(void *c, size_t idx, double re, double im) {
        reinterpret_cast<double2 *>(c)[idx] = make_double2(re, im);
    }
};
template <> struct Out<kF32> {
    static __device__ inline void put(void *c, size_t idx, double re, double im) {
        reinterpret_cast<float2 *>(c)[idx] = make_float2((float)re, (float)im);
    }
};

// MODE 0: ZGEMM / CGEMM output.  MODE 3: exact Gaussian integers (int64).
// MODE 4: residue hook (per-modulus 2M post output).
template <int T, int MODE, ElemType OT>
__global__ __launch_bounds__(256) void crt_kernel(CrtArgs a, CrtParams cp) {
    const int mblocks = (a.m + 1023) / 1024;
    const int j = blockIdx.x / mblocks;
    const int i0 = ((blockIdx.x % mblocks) * 256 + threadIdx.x) * 4;
    if (i0 >= a.m) return;
    const int8_t *base = a.res + (size_t)j * a.ldr + i0;

    if (MODE == 4) {
        for (int l = 0; l < a.rp.n; ++l) {
            const uint32_t wp = *reinterpret_cast<const uint32_t *>(base + (size_t)(2 * l) * a.plane_bytes);
            const uint32_t wm = *reinterpret_cast<const uint32_t *>(base + (size_t)(2 * l + 1) * a.plane_bytes);
            const int m = a.rp.mod[l], s = a.rp.root[l], half = (m + 1) / 2;
            int8_t *out = reinterpret_cast<int8_t *>(a.c);
            for (int e = 0; e < 4 && i0 + e < a.m; ++e) {
                const int rp = sext8(wp, e), rm = sext8(wm, e);
                int re = ((half * (rm + rp)) % m + m) % m;
                int im = ((s * ((half * (rm - rp)) % m)) % m + m) % m;
                if (re > (m - 1) / 2) re -= m;
                if (im > (m - 1) / 2) im -= m;
                const size_t o = (size_t)j * a.m + i0 + e;
                out[(size_t)(2 * l) * a.m * a.n + o] = (int8_t)re;
                out[(size_t)(2 * l + 1) * a.m * a.n + o] = (int8_t)im;
            }
        }
        return;
    }

    double sre[4][T], sim[4][T];
#pragma unroll
    for (int e = 0; e < 4; ++e)
#pragma unroll
        for (int t = 0; t < T; ++t) { sre[e][t] = 0.0; sim[e][t] = 0.0; }

    for (int l = 0; l < cp.n; ++l) {
        const uint32_t wp = *reinterpret_cast<const uint32_t *>(base + (size_t)(2 * l) * a.plane_bytes);
        const uint32_t wm = *reinterpret_cast<const uint32_t *>(base + (size_t)(2 * l + 1) * a.plane_bytes);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int rp = sext8(wp, e), rm = sext8(wm, e);
            const double u = (double)(rm + rp), v = (double)(rm - rp);
#pragma unroll
            for (int t = 0; t < T; ++t) {
                sre[e][t] = fma(u, cp.wre[l][t], sre[e][t]);
                sim[e][t] = fma(v, cp.wim[l][t], sim[e][t]);
            }
        }
    }

#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const int i = i0 + e;
        if (i >= a.m) break;
        const U192 vre = lift<T>(sre[e], cp);
        const U192 vim = lift<T>(sim[e], cp);
        if (MODE == 3) {
            // exact Gaussian integers: M < 2^63, fix the lift into [-h, h]
            int64_t re = (int64_t)vre.w0, im = (int64_t)vim.w0;
            const int64_t M = (int64_t)cp.m_lo, h = (int64_t)cp.h_lo;
            if (re > h) re -= M; else if (re < -h) re += M;
            if (im > h) im -= M; else if (im < -h) im += M;
            int64_t *out = reinterpret_cast<int64_t *>(a.c) + 2 * ((size_t)i + (size_t)j * a.ldc);
            out[0] = re;
            out[1] = im;
            // bound check: 2k max|A_i| max|B_j| <= h
            const double ma = __longlong_as_double((long long)a.amaxA[i]);
            const double mb = __longlong_as_double((long long)a.amaxB[j]);
            const unsigned __int128 need = (unsigned __int128)(2ull * (uint64_t)a.k) *
                                           (unsigned __int128)((uint64_t)ma * (uint64_t)mb);
            if (need > (unsigned __int128)(uint64_t)h) atomicOr(a.status, kStatusOverflow);
        } else {
            const int ei = a.E[i], fj = a.F[j];
            double re, im;
            if (ei == INT32_MIN || fj == INT32_MIN) {
                re = __builtin_nan("");
                im = re;
            } else {
                const int sc = ei + fj + a.scale_bias;
                re = round_scaled(vre, sc);
                im = round_scaled(vim, sc);
            }
            Out<OT>::put(a.c, (size_t)i + (size_t)j * a.ldc, re, im);
        }
    }
}

// HERK / SYRK: plane l holds C+ = A+ A-^T; C- = C+^T (Section 5), so the
// entry (i, j) needs C+ at (i, j) and at (j, i).  A workgroup owns a 32 x 32
// tile of the lower triangle and stages both tiles of every plane in LDS.
template <int T, bool REAL_ONLY>
__global__ __launch_bounds__(256) void crt_sym_kernel(CrtArgs a, CrtParams cp) {
    __shared__ __attribute__((aligned(16))) int8_t tp[2][32 * 32];
    __shared__ __attribute__((aligned(16))) int8_t tq[2][32 * 32];
    const int nb = (a.n + 31) / 32;
    const int I = blockIdx.x % nb, J = blockIdx.x / nb;
    if (I < J) return;  // strictly upper tiles: nothing to write
    const int tid = threadIdx.x;
    const int jl = tid >> 3, il0 = (tid & 7) * 4;

    double sre[4][T], sim[4][T];
#pragma unroll
    for (int e = 0; e < 4; ++e)
#pragma unroll
        for (int t = 0; t < T; ++t) { sre[e][t] = 0.0; sim[e][t] = 0.0; }

    for (int l = 0; l < cp.n; ++l) {
        const int buf = l & 1;
        const int8_t *plane = a.res + (size_t)l * a.plane_bytes;
        if (tid < 64) {          // P = C+[I rows, J cols]
            const int c = tid >> 1, h = tid & 1;
            *reinterpret_cast<uint4 *>(&tp[buf][c * 32 + h * 16]) =
                *reinterpret_cast<const uint4 *>(plane + (size_t)(J * 32 + c) * a.ldr + I * 32 + h * 16);
        } else if (tid < 128) {  // Q = C+[J rows, I cols]
            const int c = (tid - 64) >> 1, h = tid & 1;
            *reinterpret_cast<uint4 *>(&tq[buf][c * 32 + h * 16]) =
                *reinterpret_cast<const uint4 *>(plane + (size_t)(I * 32 + c) * a.ldr + J * 32 + h * 16);
        }
        __syncthreads();
        const uint32_t wp = *reinterpret_cast<const uint32_t *>(&tp[buf][jl * 32 + il0]);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int rp = sext8(wp, e);                       // C+[i, j]
            const int rm = (int)tq[buf][(il0 + e) * 32 + jl];  // C-[i, j] = C+[j, i]
            const double u = (double)(rm + rp), v = (double)(rm - rp);
#pragma unroll
            for (int t = 0; t < T; ++t) {
                sre[e][t] = fma(u, cp.wre[l][t], sre[e][t]);
                if (!REAL_ONLY) sim[e][t] = fma(v, cp.wim[l][t], sim[e][t]);
            }
        }
    }

    const int j = J * 32 + jl;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const int i = I * 32 + il0 + e;
        if (i >= a.n || j >= a.n || i < j) continue;
        const int ei = a.E[i], ej = a.E[j];
        const bool bad = ei == INT32_MIN || ej == INT32_MIN;
        const int sc = ei + ej + a.scale_bias;
        if (REAL_ONLY) {
            const double re = bad ? __builtin_nan("") : round_scaled(lift<T>(sre[e], cp), sc);
            reinterpret_cast<double *>(a.c)[(size_t)i + (size_t)j * a.ldc] = re;
        } else {
            const double re = bad ? __builtin_nan("") : round_scaled(lift<T>(sre[e], cp), sc);
            const double im = bad ? __builtin_nan("") : round_scaled(lift<T>(sim[e], cp), sc);
            reinterpret_cast<double2 *>(a.c)[(size_t)i + (size_t)j * a.ldc] = make_double2(re, im);
        }
    }
}

template <int T>
hipError_t launch_t(int mode, ElemType ot, const CrtArgs &ca, const CrtParams &cp, hipStream_t st) {
    if (mode == 1 || mode == 2) {
        const int nb = (ca.n + 31) / 32;
        const unsigned blocks = (unsigned)nb * (unsigned)nb;
        if (mode == 1) crt_sym_kernel<T, false><<<blocks, 256, 0, st>>>(ca, cp);
        else crt_sym_kernel<T, true><<<blocks, 256, 0, st>>>(ca, cp);
        return hipGetLastError();
    }
    const long blocks = (long)((ca.m + 1023) / 1024) * ca.n;
    if (blocks > 0x7FFFFFFF) return hipErrorInvalidValue;
    if (mode == 0 && ot == kF64) crt_kernel<T, 0, kF64><<<(unsigned)blocks, 256, 0, st>>>(ca, cp);
    else if (mode == 0 && ot == kF32) crt_kernel<T, 0, kF32><<<(unsigned)blocks, 256, 0, st>>>(ca, cp);
    else if (mode == 3) crt_kernel<T, 3, kF64><<<(unsigned)blocks, 256, 0, st>>>(ca, cp);
    else if (mode == 4) crt_kernel<T, 4, kF64><<<(unsigned)blocks, 256, 0, st>>>(ca, cp);
    else return hipErrorInvalidValue;
    return hipGetLastError();
}

}  // namespace

hipError_t launch_crt(int mode, ElemType out_type, const CrtArgs &ca, const CrtParams &cp, hipStream_t st) {
    if (ca.m <= 0 || ca.n <= 0) return hipSuccess;
    switch (cp.limbs) {
    case 2: return launch_t<2>(mode, out_type, ca, cp, st);
    case 3: return launch_t<3>(mode, out_type, ca, cp, st);
    case 4: return launch_t<4>(mode, out_type, ca, cp, st);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace o2m
