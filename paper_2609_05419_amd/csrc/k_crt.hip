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
// and step 7 rounds c 2^(E_i + F_j - pA - pB) once, to nearest with ties to
// even, into the output type (fp64: the limbs carried into balanced digits,
// the top two added once with an exact check of the tie against the rest,
// subnormal results from the exact multiword integer; fp32: the limb sum
// rounded to odd in fp64, then to fp32: crt_round.h).
//
// Hybrid sets (Section 3.2): for the 3M moduli the GEMM left T1 = Ar Br,
// T2 = Ai Bi, T3 = (Ar + Ai)(Br + Bi) mod m, so u = T1 - T2 and
// v = T3 - T1 - T2 enter the same limb sums with the plain CRT weights.
//
// Bound: HBM.  Algorithmic bytes per output entry: 2N residues read + 16
// written (complex fp64; 8 for complex fp32).
#include "o2m_internal.h"
#include "crt_round.h"
#include "sym_schedule.h"

#include <type_traits>

namespace o2m {
namespace {

__device__ inline int sext8(uint32_t w, int e) { return (int)(int8_t)(w >> (8 * e)); }

// One output entry in its stored type.
template <ElemType OT> struct OutT { typedef double2 type; };
template <> struct OutT<kF32> { typedef float2 type; };

// Step 7 for both components of one entry: RN(c 2^sc) into the output type,
// one rounding (fp32: never through an fp64 rounding first); NaN for a
// non-finite row or column.
template <int T, ElemType OT>
__device__ inline typename OutT<OT>::type finish(const double (&sre)[T], const double (&sim)[T],
                                                 const CrtParams &cp, bool bad, int sc) {
    if constexpr (OT == kF32) {
        if (bad) return make_float2(__builtin_nanf(""), __builtin_nanf(""));
        return make_float2(lift_round_f32<T>(sre, cp.mlimb, cp.inv_m, sc),
                           lift_round_f32<T>(sim, cp.mlimb, cp.inv_m, sc));
    } else {
        if (bad) return make_double2(__builtin_nan(""), __builtin_nan(""));
        return make_double2(lift_round<T>(sre, cp.mlimb, cp.inv_m, sc), lift_round<T>(sim, cp.mlimb, cp.inv_m, sc));
    }
}

// MODE 0: ZGEMM / CGEMM output.  MODE 3: exact Gaussian integers (int64).
// MODE 4: residue hook (per-modulus 2M post output).  Each thread owns R = 4
// consecutive rows of one column: one dword per plane.  Up to three limbs
// the row exponents are fetched before the limb sums and the kernel is held
// to 80 registers (six waves per SIMD; it needs 81 otherwise); with more
// limbs both would cost occupancy or spills, and the exponents are read when
// the rows are finished.
template <int T, int MODE, ElemType OT>
__global__ __launch_bounds__(256, T <= 3 ? 6 : 1) void crt_kernel(CrtArgs a, CrtParams cp) {
    constexpr int R = 4;
    const int rows_per_block = 256 * R;
    const int mblocks = (a.m + rows_per_block - 1) / rows_per_block;
    const int j = blockIdx.x / mblocks;
    const int i0 = ((blockIdx.x % mblocks) * 256 + threadIdx.x) * R;
    // complex outputs pass through LDS in their stored type (each wave its own
    // 256 entries) and leave in row order, so a lane may store rows of another
    // lane: a wave leaves only when all its rows are beyond m, and a lane
    // beyond m reads row 0 instead (its sums are never stored)
    constexpr bool STAGE = MODE == 0;
    typedef typename OutT<OT>::type SV;
    __shared__ SV stage[STAGE ? 256 * R : 1];
    const int lane = threadIdx.x & 63, w0 = threadIdx.x & ~63;
    if ((STAGE ? i0 - lane * R : i0) >= a.m) return;
    const int8_t *base = a.res + (size_t)j * a.ldr + (i0 < a.m ? i0 : 0);

    if (MODE == 4) {
        for (int l = 0; l < cp.n; ++l) {
            const int m = a.hmod[l], s = a.hroot[l], half = (m + 1) / 2;
            int8_t *out = reinterpret_cast<int8_t *>(a.c);
            for (int e = 0; e < R && i0 + e < a.m; ++e) {
                int re, im;
                if (l < cp.n2) {   // 2M post (eq. 2m-post)
                    const int rp = base[(size_t)(2 * l) * a.plane_bytes + e];
                    const int rm = base[(size_t)(2 * l + 1) * a.plane_bytes + e];
                    re = ((half * (rm + rp)) % m + m) % m;
                    im = ((s * ((half * (rm - rp)) % m)) % m + m) % m;
                } else {           // 3M post
                    const size_t p0 = (size_t)(2 * cp.n2 + 3 * (l - cp.n2));
                    const int t1 = base[p0 * a.plane_bytes + e];
                    const int t2 = base[(p0 + 1) * a.plane_bytes + e];
                    const int t3 = base[(p0 + 2) * a.plane_bytes + e];
                    re = ((t1 - t2) % m + m) % m;
                    im = ((t3 - t1 - t2) % m + 2 * m) % m;
                }
                if (re > (m - 1) / 2) re -= m;
                if (im > (m - 1) / 2) im -= m;
                const size_t o = (size_t)j * a.m + i0 + e;
                out[(size_t)(2 * l) * a.m * a.n + o] = (int8_t)re;
                out[(size_t)(2 * l + 1) * a.m * a.n + o] = (int8_t)im;
            }
        }
        return;
    }

    // the exponents of the thread's rows and column, fetched before the limb
    // sums so that their latency is hidden behind them (E holds every padded
    // row, and i0, a multiple of 4, is below m or replaced by row 0)
    constexpr bool EARLY = MODE == 0 && T <= 3;
    int ev[R] = {}, fj = 0;
    if constexpr (EARLY) {
        const int4 e4 = *reinterpret_cast<const int4 *>(a.E + (i0 < a.m ? i0 : 0));
        ev[0] = e4.x; ev[1] = e4.y; ev[2] = e4.z; ev[3] = e4.w;
        fj = a.F[j];
    }

    double sre[R][T], sim[R][T];
#pragma unroll
    for (int e = 0; e < R; ++e)
#pragma unroll
        for (int t = 0; t < T; ++t) { sre[e][t] = 0.0; sim[e][t] = 0.0; }

    // 2M moduli, in chunks whose plane loads are all issued before their limb
    // sums, so that each wave keeps several loads in flight
    auto chunk2m = [&](int l0, auto ch) {
        constexpr int CH = decltype(ch)::value;
        uint32_t wp[CH], wm[CH];
#pragma unroll
        for (int c = 0; c < CH; ++c) {
            wp[c] = *reinterpret_cast<const uint32_t *>(base + (size_t)(2 * (l0 + c)) * a.plane_bytes);
            wm[c] = *reinterpret_cast<const uint32_t *>(base + (size_t)(2 * (l0 + c) + 1) * a.plane_bytes);
        }
#pragma unroll
        for (int c = 0; c < CH; ++c)
#pragma unroll
            for (int e = 0; e < R; ++e) {
                const int rp = sext8(wp[c], e), rm = sext8(wm[c], e);
                const double u = (double)(rm + rp), v = (double)(rm - rp);
#pragma unroll
                for (int t = 0; t < T; ++t) {
                    sre[e][t] = fma(u, cp.wre[l0 + c][t], sre[e][t]);
                    sim[e][t] = fma(v, cp.wim[l0 + c][t], sim[e][t]);
                }
            }
    };
    int l = 0;
    for (; l + 8 <= cp.n2; l += 8) chunk2m(l, std::integral_constant<int, 8>());
    if (l + 4 <= cp.n2) {
        chunk2m(l, std::integral_constant<int, 4>());
        l += 4;
    }
    for (; l < cp.n2; ++l) chunk2m(l, std::integral_constant<int, 1>());
    // 3M moduli of a hybrid set: Re = T1 - T2, Im = T3 - T1 - T2, plain
    // weights; loads issued per chunk as above
    auto chunk3m = [&](int l0, auto ch) {
        constexpr int CH = decltype(ch)::value;
        uint32_t w[CH][3];
#pragma unroll
        for (int c = 0; c < CH; ++c) {
            const size_t p0 = (size_t)(2 * cp.n2 + 3 * (l0 + c - cp.n2));
#pragma unroll
            for (int q = 0; q < 3; ++q) w[c][q] = *reinterpret_cast<const uint32_t *>(base + (p0 + q) * a.plane_bytes);
        }
#pragma unroll
        for (int c = 0; c < CH; ++c)
#pragma unroll
            for (int e = 0; e < R; ++e) {
                const int t1 = sext8(w[c][0], e), t2 = sext8(w[c][1], e), t3 = sext8(w[c][2], e);
                const double u = (double)(t1 - t2), v = (double)(t3 - t1 - t2);
#pragma unroll
                for (int t = 0; t < T; ++t) {
                    sre[e][t] = fma(u, cp.wre[l0 + c][t], sre[e][t]);
                    sim[e][t] = fma(v, cp.wre[l0 + c][t], sim[e][t]);
                }
            }
    };
    for (; l + 2 <= cp.n; l += 2) chunk3m(l, std::integral_constant<int, 2>());
    for (; l < cp.n; ++l) chunk3m(l, std::integral_constant<int, 1>());

#pragma unroll
    for (int e = 0; e < R; ++e) {
        const int i = i0 + e;
        if (i >= a.m) break;
        if constexpr (MODE == 3) {
            const auto vre = lift_exact<T>(sre[e], cp.mlimb, cp.inv_m);
            const auto vim = lift_exact<T>(sim[e], cp.mlimb, cp.inv_m);
            // exact Gaussian integers: M < 2^63, fix the lift into [-h, h]
            int64_t re = (int64_t)vre.w[0], im = (int64_t)vim.w[0];
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
            const int ei = EARLY ? ev[e] : a.E[i];
            if constexpr (!EARLY) fj = a.F[j];
            const SV v = finish<T, OT>(sre[e], sim[e], cp, ei == INT32_MIN || fj == INT32_MIN, ei + fj + a.scale_bias);
            if constexpr (STAGE) stage[threadIdx.x * R + e] = v;
            else reinterpret_cast<SV *>(a.c)[(size_t)i + (size_t)j * a.ldc] = v;
        }
    }
    if constexpr (STAGE) {
        // the wave's 256 rows leave in row order, 64 consecutive rows per store
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
        const int ib = (blockIdx.x % mblocks) * rows_per_block + w0 * R;
#pragma unroll
        for (int e = 0; e < R; ++e) {
            const int i = ib + e * 64 + lane;
            const SV v = stage[w0 * R + e * 64 + lane];
            if (i < a.m) reinterpret_cast<SV *>(a.c)[(size_t)i + (size_t)j * a.ldc] = v;
        }
    }
}

// HERK / SYRK: plane l holds C+ = A+ A-^T; C- = C+^T (Section 5), so the
// entry (i, j) needs C+ at (i, j) and at (j, i).  A workgroup owns a 32 x 32
// tile of the lower triangle and stages both tiles of CH planes at a time in
// LDS; the next CH planes' copies are in flight while these planes' limb sums
// run.  The real-only form, light on arithmetic, waits on memory and takes 8
// planes per chunk; the complex form issues twice the limb sums and takes 4,
// whose staging registers cost less occupancy (measured: 8 planes or copies
// straight into LDS were slower for it).  The rows' exponents are fetched
// before the limb sums; the complex form is held to 80 registers up to three
// limbs (six waves per SIMD) and 96 with four (five).
template <int T, bool REAL_ONLY>
__global__ __launch_bounds__(256, REAL_ONLY ? 1 : (T <= 3 ? 6 : 5)) void crt_sym_kernel(CrtArgs a, CrtParams cp) {
    constexpr int CH = REAL_ONLY ? 8 : 4;  // planes per chunk
    // [plane of the chunk][P = C+ tile (I, J), Q = C+ tile (J, I)], column-major 32 x 32
    __shared__ __attribute__((aligned(16))) int8_t tl[CH][2][32 * 32];
    const SymTile st = sym_tile_of(blockIdx.x, (a.n + 31) / 32);
    if (!st.valid) return;  // idle slot or strictly upper tile: nothing to write
    // tile (I, J) of the lower triangle, or its mirror (J, I) for the upper:
    // entry (i, j) needs C+ at (i, j) and (j, i) either way, and the same
    // coalesced layout writes it
    const int I = a.upper ? st.J : st.I, J = a.upper ? st.I : st.J;
    const int tid = threadIdx.x;
    // the thread's entries: rows r0 + 8e (e = 0..3) of column jl, so that each
    // store writes whole 128-byte lines across 8 lanes
    const int jl = tid >> 3, r0 = tid & 7;

    // each thread copies 16 bytes (half a column of P or of Q) of the chunk's
    // planes of one parity: planes l0 + po, l0 + po + 2, ..
    const int pc = tid & 127, po = tid >> 7;
    const int q = pc >> 6, c = (pc & 63) >> 1, h = pc & 1;
    const int8_t *src = a.res + (q == 0 ? (size_t)(J * 32 + c) * a.ldr + I * 32 + h * 16
                                        : (size_t)(I * 32 + c) * a.ldr + J * 32 + h * 16);
    const int dst = c * 32 + h * 16;

    // the exponents of the thread's rows and column, fetched before the limb
    // sums (E holds every padded row, and the tiles cover no more)
    int ev[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) ev[e] = a.E[I * 32 + r0 + 8 * e];
    const int ej = a.E[J * 32 + jl];

    double sre[4][T], sim[4][T];
#pragma unroll
    for (int e = 0; e < 4; ++e)
#pragma unroll
        for (int t = 0; t < T; ++t) { sre[e][t] = 0.0; sim[e][t] = 0.0; }

    // every copy is taken, from plane n - 1 past the last one (never summed),
    // so that none waits inside a branch; the chunk is held in one vector
    // value, which stays in registers
    typedef unsigned int Stage __attribute__((ext_vector_type(2 * CH)));
    Stage nx;
    auto fetch = [&](int l0) {
#pragma unroll
        for (int x = 0; x < CH / 2; ++x) {
            const int l = min(l0 + po + 2 * x, cp.n - 1);
            const uint4 w = *reinterpret_cast<const uint4 *>(src + (size_t)l * a.plane_bytes);
            nx[4 * x] = w.x;
            nx[4 * x + 1] = w.y;
            nx[4 * x + 2] = w.z;
            nx[4 * x + 3] = w.w;
        }
    };
    fetch(0);
    for (int l0 = 0; l0 < cp.n; l0 += CH) {
        if (l0 > 0) __syncthreads();  // the previous chunk's reads are done
#pragma unroll
        for (int x = 0; x < CH / 2; ++x)
            *reinterpret_cast<uint4 *>(&tl[po + 2 * x][q][dst]) =
                make_uint4(nx[4 * x], nx[4 * x + 1], nx[4 * x + 2], nx[4 * x + 3]);
        __syncthreads();
        if (l0 + CH < cp.n) fetch(l0 + CH);
        asm volatile("" ::: "memory");  // the next chunk's loads stay ahead of the sums
#pragma unroll
        for (int t = 0; t < CH; ++t) {
            const int l = l0 + t;
            if (l >= cp.n) break;  // uniform
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int rp = (int)tl[t][0][jl * 32 + r0 + 8 * e];    // C+[i, j]
                const int rm = (int)tl[t][1][(r0 + 8 * e) * 32 + jl];  // C-[i, j] = C+[j, i]
                const double u = (double)(rm + rp), v = (double)(rm - rp);
#pragma unroll
                for (int k = 0; k < T; ++k) {
                    sre[e][k] = fma(u, cp.wre[l][k], sre[e][k]);
                    if (!REAL_ONLY) sim[e][k] = fma(v, cp.wim[l][k], sim[e][k]);
                }
            }
        }
    }

    const int j = J * 32 + jl;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const int i = I * 32 + r0 + 8 * e;
        if (i >= a.n || j >= a.n || (a.upper ? i > j : i < j)) continue;
        const int ei = ev[e];
        const bool bad = ei == INT32_MIN || ej == INT32_MIN;
        const int sc = ei + ej + a.scale_bias;
        if (REAL_ONLY) {
            const double re = bad ? __builtin_nan("") : lift_round<T>(sre[e], cp.mlimb, cp.inv_m, sc);
            reinterpret_cast<double *>(a.c)[(size_t)i + (size_t)j * a.ldc] = re;
        } else {
            const double re = bad ? __builtin_nan("") : lift_round<T>(sre[e], cp.mlimb, cp.inv_m, sc);
            const double im = bad ? __builtin_nan("") : lift_round<T>(sim[e], cp.mlimb, cp.inv_m, sc);
            reinterpret_cast<double2 *>(a.c)[(size_t)i + (size_t)j * a.ldc] = make_double2(re, im);
        }
    }
}

template <int T>
hipError_t launch_t(int mode, ElemType ot, const CrtArgs &ca, const CrtParams &cp, hipStream_t st) {
    if (mode == 1 || mode == 2) {
        // symmetric ops: 2M moduli only, so at most 22 moduli and four limbs
        if constexpr (T > 4) {
            return hipErrorInvalidValue;
        } else {
            if (cp.n2 != cp.n) return hipErrorInvalidValue;
            const long blocks = sym_grid((ca.n + 31) / 32);
            if (blocks > 0x7FFFFFFF) return hipErrorInvalidValue;
            if (mode == 1) crt_sym_kernel<T, false><<<(unsigned)blocks, 256, 0, st>>>(ca, cp);
            else crt_sym_kernel<T, true><<<(unsigned)blocks, 256, 0, st>>>(ca, cp);
            return hipGetLastError();
        }
    }
    // 4 rows of one column per thread, 1024 rows per workgroup
    const long blocks = (long)((ca.m + 1023) / 1024) * ca.n;
    if (blocks > 0x7FFFFFFF) return hipErrorInvalidValue;
    if (mode == 0 && ot == kF64) crt_kernel<T, 0, kF64><<<(unsigned)blocks, 256, 0, st>>>(ca, cp);
    else if (mode == 0 && ot == kF32) crt_kernel<T, 0, kF32><<<(unsigned)blocks, 256, 0, st>>>(ca, cp);
    else if (mode == 3 && T == 2) crt_kernel<2, 3, kF64><<<(unsigned)blocks, 256, 0, st>>>(ca, cp);
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
    case 5: return launch_t<5>(mode, out_type, ca, cp, st);
    case 6: return launch_t<6>(mode, out_type, ca, cp, st);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace o2m
