// K1: scaling exponents (Algorithm 1, step 2).
//
// The row scale of A and the column scale of B are powers of two,
// sigma_i = 2^(E_i - pA), tau_j = 2^(F_j - pB), with E_i the frexp exponent
// of the largest |Re| or |Im| in row i (so that max < 2^E_i).  The maxima are
// found with atomicMax on the bit patterns of |x| (for non-negative doubles
// the bit pattern is monotone in the value, and Inf/NaN patterns sit above
// every finite one, which flags non-finite rows for free).
//
// Cauchy-Schwarz rule (the paper leaves sigma, tau open and points to norm
// based rules of the Ozaki-II literature): the 2-norm of every row / column is
// bounded by 2^G with an exact integer sum of squares of the parts rounded up
// to 2^-20 of the row maximum.  One pass over the operand finds both: each
// chunk of a row is reduced against its own maximum (cs_scan_*), and a
// combine step brackets the row's exact sum from the chunks' (cs_bounds.h),
// settles G, and sums the rare row whose bracket straddles a power of 4 again
// from the data (cs_combine_kernel).
//
// Bound: HBM.  Algorithmic bytes = the matrix read once per pass (16 B per
// complex fp64 element).  Rows of a column-major A are strided, so a thread owns one
// row and walks a chunk of columns: every load instruction of a wave reads 64
// consecutive rows (1 KB contiguous).  Columns of B are contiguous: a block
// owns a chunk of one column.
#include "o2m_internal.h"
#include "cs_bounds.h"

namespace o2m {
namespace {

__device__ inline unsigned long long bits_of(double x) {
    // |x| as a bit pattern: monotone in |x| for finite values, and every NaN
    // (of either sign) sorts above +Inf once the sign bit is cleared
    return (unsigned long long)__double_as_longlong(x) & 0x7FFFFFFFFFFFFFFFull;
}

__device__ inline unsigned long long umax(unsigned long long a, unsigned long long b) { return a > b ? a : b; }

// A NaN in either part of an entry wins the maximum (fmax would drop it):
// bits() takes the larger bit pattern of |Re| and |Im|.
// An entry as loaded, and what the two passes compute from it.  In column
// mode a thread issues the loads of its kBatch rows of the chunk before using
// any (a workgroup then reads 32 KB of one column at once).
// The scaling kernels read each operand entry once, and the residue pass
// reads it again next.  For large operands (beyond what the 256 MB Infinity
// Cache could keep for that pass) the loads are non-temporal (NT: no cache
// allocation), which measured 11-14% faster on 8192 x 8192 complex fp64
// operands (10% at 4096 x 4096); smaller ones keep plain loads, which leave
// them cached for the residue pass (at 2048 x 2048 non-temporal scans made
// that pass 4-7% slower).
template <bool NT, typename T> __device__ inline T ld1(const T *p) {
    if constexpr (NT) return __builtin_nontemporal_load(p);
    else return *p;
}
constexpr size_t kStreamBytes = size_t(128) << 20;   // operands from 128 MiB stream

template <ElemType ET> struct Raw;
template <> struct Raw<kF64> {
    typedef double2 T;
    static constexpr int n = 2;
    template <bool NT = false> static __device__ inline T load(const void *X, size_t idx) {
        const double2 *q = reinterpret_cast<const double2 *>(X) + idx;
        return make_double2(ld1<NT>(&q->x), ld1<NT>(&q->y));
    }
    static __device__ inline T zero() { return make_double2(0.0, 0.0); }
    static __device__ inline unsigned long long bits(T v) { return umax(bits_of(v.x), bits_of(v.y)); }
    static __device__ inline void parts(T v, double (&p)[2]) { p[0] = v.x; p[1] = v.y; }
};
template <> struct Raw<kF32> {
    typedef float2 T;
    static constexpr int n = 2;
    template <bool NT = false> static __device__ inline T load(const void *X, size_t idx) {
        const float2 *q = reinterpret_cast<const float2 *>(X) + idx;
        return make_float2(ld1<NT>(&q->x), ld1<NT>(&q->y));
    }
    static __device__ inline T zero() { return make_float2(0.0f, 0.0f); }
    static __device__ inline unsigned long long bits(T v) { return umax(bits_of((double)v.x), bits_of((double)v.y)); }
    static __device__ inline void parts(T v, double (&p)[2]) { p[0] = (double)v.x; p[1] = (double)v.y; }
};
template <> struct Raw<kI32> {  // Gaussian integers: maxima only
    typedef int2 T;
    template <bool NT = false> static __device__ inline T load(const void *X, size_t idx) {
        const int2 *q = reinterpret_cast<const int2 *>(X) + idx;
        return make_int2(ld1<NT>(&q->x), ld1<NT>(&q->y));
    }
    static __device__ inline T zero() { return make_int2(0, 0); }
    static __device__ inline unsigned long long bits(T v) { return umax(bits_of((double)v.x), bits_of((double)v.y)); }
};
template <> struct Raw<kR64> {
    typedef double T;
    static constexpr int n = 1;
    template <bool NT = false> static __device__ inline T load(const void *X, size_t idx) {
        return ld1<NT>(reinterpret_cast<const double *>(X) + idx);
    }
    static __device__ inline T zero() { return 0.0; }
    static __device__ inline unsigned long long bits(T v) { return bits_of(v); }
    static __device__ inline void parts(T v, double (&p)[2]) { p[0] = v; p[1] = 0.0; }
};

constexpr int kBatch = 8;   // loads issued together per thread (column mode)

constexpr int kRowChunk = 128;    // columns per thread in row mode (at most)
constexpr int kColChunk = 2048;   // rows per block in column mode

template <ElemType ET, bool NT>
__global__ __launch_bounds__(256) void amax_rows(int rows, int cols, int chunk, const void *X, int ld,
                                                 unsigned long long *amax) {
    const int r = blockIdx.x * 256 + threadIdx.x;
    if (r >= rows) return;
    const int c0 = blockIdx.y * chunk;
    const int c1 = min(cols, c0 + chunk);
    unsigned long long best = 0;
    // one load in flight per thread: a workgroup's waves walk one column (4 KB
    // contiguous) at a time; batching loads over columns opened more DRAM
    // pages at once and measured slower at 8192^2 (faster only at 4096^2)
    for (int c = c0; c < c1; ++c) best = umax(best, Raw<ET>::bits(Raw<ET>::template load<NT>(X, (size_t)r + (size_t)c * ld)));
    if (best) atomicMax(amax + r, best);
}

template <ElemType ET, bool NT>
__global__ __launch_bounds__(256) void amax_cols(int rows, int cols, const void *X, int ld,
                                                 unsigned long long *amax) {
    const int c = blockIdx.x;
    const int r0 = blockIdx.y * kColChunk;
    const int r1 = min(rows, r0 + kColChunk);
    unsigned long long best = 0;
    static_assert(kColChunk == 256 * kBatch, "one batch of loads per thread covers the chunk");
    typename Raw<ET>::T v[kBatch];
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
        const int r = r0 + threadIdx.x + 256 * u;
        v[u] = r < r1 ? Raw<ET>::template load<NT>(X, (size_t)r + (size_t)c * ld) : Raw<ET>::zero();
    }
#pragma unroll
    for (int u = 0; u < kBatch; ++u) best = umax(best, Raw<ET>::bits(v[u]));
    // wave reduction, then one atomic per wave
    for (int off = 32; off > 0; off >>= 1) {
        unsigned long long o = __shfl_xor(best, off, 64);
        best = o > best ? o : best;
    }
    if ((threadIdx.x & 63) == 0 && best) atomicMax(amax + c, best);
}

// ---- Cauchy-Schwarz rule, one pass --------------------------------------
// Per (row, chunk) record: the chunk's max bit pattern, S2 = sum y^2,
// S1 = sum y and n = #nonzero parts, with y = max(1, ceil(|v| 2^(20 - e))) for
// the chunk's max exponent e (packed S1 | n << 44: S1 < 2^33, n < 2^13).
constexpr int kS1Bits = 44;

template <ElemType ET>
__device__ inline void cs_accumulate(typename Raw<ET>::T x, int e, unsigned long long &s2, unsigned long long &s1,
                                     unsigned long long &n) {
    double v[2];
    Raw<ET>::parts(x, v);
#pragma unroll
    for (int q = 0; q < Raw<ET>::n; ++q) {
        if (v[q] == 0.0) continue;
        double u = ceil(ldexp(fabs(v[q]), 20 - e));
        u = u < 1.0 ? 1.0 : u;
        const unsigned long long y = (unsigned long long)u;
        s2 += y * y;
        s1 += y;
        n += 1;
    }
}

// The exponent e of a finite nonzero max bit pattern (max < 2^e).
__device__ inline int exponent_of(unsigned long long b) {
    int e;
    frexp(__longlong_as_double((long long)b), &e);
    return e;
}

// Row mode (rows of a column-major X): a workgroup covers 64 rows x 4 CPT
// columns, wave w the columns [w CPT, (w + 1) CPT) of the chunk, so that every
// load of a wave reads 64 consecutive rows of one column (1 KB).  A thread
// holds its CPT entries while the four waves agree on each row's chunk
// maximum through LDS, then sums against it.  Loads are clamped into the
// matrix and their values dropped beyond it, so all of them can be in flight.
template <ElemType ET, int CPT, bool NT>
__global__ __launch_bounds__(256) void cs_scan_rows(int rows, int cols, const void *X, int ld, CsPartials p,
                                                    int chunk_ofs) {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int r = blockIdx.x * 64 + lane;
    const int rc = r < rows ? r : rows - 1;
    const int c0 = blockIdx.y * 4 * CPT + w * CPT;
    typename Raw<ET>::T v[CPT];
#pragma unroll
    for (int u = 0; u < CPT; ++u) {
        const int c = c0 + u < cols ? c0 + u : cols - 1;
        v[u] = Raw<ET>::template load<NT>(X, (size_t)rc + (size_t)c * ld);
    }
#pragma unroll
    for (int u = 0; u < CPT; ++u)
        if (c0 + u >= cols) v[u] = Raw<ET>::zero();
    unsigned long long best = 0;
#pragma unroll
    for (int u = 0; u < CPT; ++u) best = umax(best, Raw<ET>::bits(v[u]));

    __shared__ unsigned long long smax[4][64], ss2[4][64], ss1[4][64], snn[4][64];
    smax[w][lane] = best;
    __syncthreads();
    best = umax(umax(smax[0][lane], smax[1][lane]), umax(smax[2][lane], smax[3][lane]));
    unsigned long long s2 = 0, s1 = 0, n = 0;
    if (best != 0 && best < 0x7FF0000000000000ull) {
        const int e = exponent_of(best);
#pragma unroll
        for (int u = 0; u < CPT; ++u) cs_accumulate<ET>(v[u], e, s2, s1, n);
    }
    ss2[w][lane] = s2;
    ss1[w][lane] = s1;
    snn[w][lane] = n;
    __syncthreads();
    if (w == 0 && r < rows) {
        s2 = ss2[0][lane] + ss2[1][lane] + ss2[2][lane] + ss2[3][lane];
        s1 = ss1[0][lane] + ss1[1][lane] + ss1[2][lane] + ss1[3][lane];
        n = snn[0][lane] + snn[1][lane] + snn[2][lane] + snn[3][lane];
        const size_t idx = (size_t)(chunk_ofs + blockIdx.y) * p.pitch + r;
        p.mx[idx] = best;
        p.s2[idx] = s2;
        p.s1n[idx] = s1 | (n << kS1Bits);
    }
}

// Column mode (columns of a column-major X, contiguous): a workgroup covers
// kColChunk entries of one column, kBatch per thread, held while the
// workgroup agrees on the chunk maximum.  PAIRS: complex fp32 entries are
// read two per 16-byte load (the host sets it when every pair is aligned).
template <ElemType ET, bool PAIRS, bool NT>
__global__ __launch_bounds__(256) void cs_scan_cols(int rows, int cols, const void *X, int ld, CsPartials p) {
    const int c = blockIdx.x;
    const int r0 = blockIdx.y * kColChunk;
    const int r1 = min(rows, r0 + kColChunk);
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    typename Raw<ET>::T x[kBatch];
    if constexpr (PAIRS) {
        static_assert(ET == kF32, "pairs of complex fp32 entries");
        const float2 *Xc = reinterpret_cast<const float2 *>(X) + (size_t)c * ld;
#pragma unroll
        for (int u = 0; u < kBatch / 2; ++u) {
            const int r = r0 + 2 * threadIdx.x + 512 * u;
            float4 v = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
            if (r + 1 < r1) {
                const float *q = reinterpret_cast<const float *>(Xc + r);
                v = make_float4(ld1<NT>(q), ld1<NT>(q + 1), ld1<NT>(q + 2), ld1<NT>(q + 3));
            } else if (r < r1) {
                const float2 t = Xc[r];
                v.x = t.x;
                v.y = t.y;
            }
            x[2 * u] = make_float2(v.x, v.y);
            x[2 * u + 1] = make_float2(v.z, v.w);
        }
    } else {
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
            const int r = r0 + threadIdx.x + 256 * u;
            x[u] = r < r1 ? Raw<ET>::template load<NT>(X, (size_t)r + (size_t)c * ld) : Raw<ET>::zero();
        }
    }
    unsigned long long best = 0;
#pragma unroll
    for (int u = 0; u < kBatch; ++u) best = umax(best, Raw<ET>::bits(x[u]));
    for (int off = 32; off > 0; off >>= 1) best = umax(best, __shfl_xor(best, off, 64));
    __shared__ unsigned long long sm[4], s[3][4];
    if (lane == 0) sm[w] = best;
    __syncthreads();
    best = umax(umax(sm[0], sm[1]), umax(sm[2], sm[3]));
    unsigned long long s2 = 0, s1 = 0, n = 0;
    if (best != 0 && best < 0x7FF0000000000000ull) {
        const int e = exponent_of(best);
#pragma unroll
        for (int u = 0; u < kBatch; ++u) cs_accumulate<ET>(x[u], e, s2, s1, n);
    }
    for (int off = 32; off > 0; off >>= 1) {
        s2 += __shfl_xor(s2, off, 64);
        s1 += __shfl_xor(s1, off, 64);
        n += __shfl_xor(n, off, 64);
    }
    if (lane == 0) {
        s[0][w] = s2;
        s[1][w] = s1;
        s[2][w] = n;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        s2 = s[0][0] + s[0][1] + s[0][2] + s[0][3];
        s1 = s[1][0] + s[1][1] + s[1][2] + s[1][3];
        n = s[2][0] + s[2][1] + s[2][2] + s[2][3];
        const size_t idx = (size_t)blockIdx.y * p.pitch + c;
        p.mx[idx] = best;
        p.s2[idx] = s2;
        p.s1n[idx] = s1 | (n << kS1Bits);
    }
}

// ceil(|v| 2^(20 - e))^2 for one part: |v| < 2^e, so the ceiling is at most
// 2^20; a nonzero part whose scaled value underflows lies in (0, 1) and
// counts as 1.
__device__ inline unsigned long long ssq_term(double v, int e) {
    if (v == 0.0) return 0ull;
    double u = ceil(ldexp(fabs(v), 20 - e));
    u = u < 1.0 ? 1.0 : u;
    const unsigned long long q = (unsigned long long)u;
    return q * q;
}

constexpr int kCombineWaves = 16;

// Combine: a workgroup takes 64 rows of A (blocks [0, ceil(ca/64))) or 64
// columns of B (the blocks after), its 16 waves every 16th chunk each.
// E = the max exponent over the chunks (INT32_MIN for Inf/NaN, which also sets
// kStatusNonfinite; 0 for a zero row), then the bracket of U from the chunk
// records settles G = E - 20 + d.  A row whose bracket straddles a power of 4
// is summed again from the data by the whole workgroup (row i of A, and of B2
// for rank-2k updates; column j of B; with transposed operands, a column of
// the stored A or a row of the stored B) against E.
template <ElemType ET>
__global__ __launch_bounds__(64 * kCombineWaves) void cs_combine_kernel(CsCombineArgs g) {
    const int ba = (g.ca + 63) / 64;
    int blk = blockIdx.x;
    const bool side_a = blk < ba;
    if (!side_a) blk -= ba;
    const CsPartials &p = side_a ? g.pa : g.pb;
    const int cnt = side_a ? g.ca : g.cb;
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int i = blk * 64 + lane;
    const int ic = i < cnt ? i : cnt - 1;
    __shared__ unsigned long long sm[kCombineWaves][64], slo[kCombineWaves][64], shi[kCombineWaves][64];
    __shared__ int sE[64];
    __shared__ unsigned long long sflag;

    unsigned long long mb = 0;
#pragma unroll 4
    for (int c = w; c < p.chunks; c += kCombineWaves) mb = umax(mb, p.mx[(size_t)c * p.pitch + ic]);
    sm[w][lane] = mb;
    __syncthreads();
#pragma unroll
    for (int q = 0; q < kCombineWaves; ++q) mb = umax(mb, sm[q][lane]);
    const bool bad = mb >= 0x7FF0000000000000ull;
    const int e = bad || mb == 0 ? 0 : exponent_of(mb);
    uint64_t lo = 0, hi = 0;
    if (!bad && mb != 0) {
#pragma unroll 4
        for (int c = w; c < p.chunks; c += kCombineWaves) {
            const size_t idx = (size_t)c * p.pitch + ic;
            const unsigned long long v = p.s1n[idx];
            const unsigned long long n = v >> kS1Bits;
            const unsigned long long x = p.mx[idx], s2 = p.s2[idx];
            if (n == 0) continue;
            uint64_t l, h;
            cs_chunk_bounds(e - exponent_of(x), s2, v & ((1ull << kS1Bits) - 1), n, &l, &h);
            lo += l;
            hi += h;
        }
    }
    slo[w][lane] = lo;
    shi[w][lane] = hi;
    __syncthreads();
    if (w == 0) {
        const bool valid = i < cnt;
        int out = e;
        bool f = false;
        if (bad) {
            out = INT32_MIN;
        } else if (mb != 0) {
            lo = hi = 0;
#pragma unroll
            for (int q = 0; q < kCombineWaves; ++q) {
                lo += slo[q][lane];
                hi += shi[q][lane];
            }
            const int d = cs_d_of(lo);
            if (d == cs_d_of(hi)) out = e + d - 20;
            else f = valid;
        }
        if (valid) (side_a ? g.Ea : g.Eb)[i] = out;
        sE[lane] = e;
        const unsigned long long seen = __ballot(valid && bad);
        if (seen != 0 && lane == __ffsll((long long)seen) - 1) atomicOr(g.status, kStatusNonfinite);
        const unsigned long long open = __ballot(f);
        if (lane == 0) sflag = open;
    }
    __syncthreads();
    // entries left open: the rule's sum from the data, all threads together
    unsigned long long open = sflag;   // uniform
    while (open) {
        const int l = __builtin_ctzll(open);
        open &= open - 1;
        const int r = blk * 64 + l, er = sE[l];
        unsigned long long acc = 0;
        auto add = [&](typename Raw<ET>::T x) {
            double v[2];
            Raw<ET>::parts(x, v);
#pragma unroll
            for (int q = 0; q < Raw<ET>::n; ++q) acc += ssq_term(v[q], er);
        };
        const void *X = side_a ? g.A : g.B;
        const int ld = side_a ? g.lda : g.ldb;
        const bool as_rows = (side_a ? g.amode : g.bmode) == 0;
        for (int c = threadIdx.x; c < g.k; c += 64 * kCombineWaves) {
            add(Raw<ET>::load(X, as_rows ? (size_t)r + (size_t)c * ld : (size_t)c + (size_t)r * ld));
            if (side_a && g.B2) add(Raw<ET>::load(g.B2, (size_t)r + (size_t)c * g.ldb2));
        }
        for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off, 64);
        if (lane == 0) sm[w][0] = acc;
        __syncthreads();
        if (threadIdx.x == 0) {
            unsigned long long U = 0;
            for (int q = 0; q < kCombineWaves; ++q) U += sm[q][0];
            (side_a ? g.Ea : g.Eb)[r] = er - 20 + cs_d_of(U);
        }
        __syncthreads();
    }
}

// Entries [0, ca) of (amax_a, Ea), then [0, cb) of (amax_b, Eb), in one launch.
// A row or column holding Inf or NaN gets E = INT32_MIN and sets the device
// status bit kStatusNonfinite (one atomic per wave that saw one).
__global__ void exponents_kernel(int ca, const unsigned long long *amax_a, int32_t *Ea, int cb,
                                 const unsigned long long *amax_b, int32_t *Eb, int *status) {
    int i = blockIdx.x * 256 + threadIdx.x;
    const unsigned long long *amax = amax_a;
    int32_t *E = Ea;
    bool valid = true;
    if (i >= ca) { i -= ca; amax = amax_b; E = Eb; valid = i < cb; }
    bool bad = false;
    if (valid) {
        const unsigned long long b = amax[i];
        int e;
        bad = b >= 0x7FF0000000000000ull;
        if (bad) e = INT32_MIN;                                // Inf or NaN in the row
        else if (b == 0) e = 0;                                // zero row: E = 0
        else frexp(__longlong_as_double((long long)b), &e);    // max < 2^e
        E[i] = e;
    }
    const unsigned long long seen = __ballot(bad);
    if (seen != 0 && (int)(threadIdx.x & 63) == __ffsll((long long)seen) - 1) atomicOr(status, kStatusNonfinite);
}

__global__ void zero_kernel(uint4 *p, size_t n16, unsigned char *tail, int ntail) {
    size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
    const size_t stride = (size_t)gridDim.x * 256;
    for (; i < n16; i += stride) p[i] = make_uint4(0, 0, 0, 0);
    if (blockIdx.x == 0 && (int)threadIdx.x < ntail) tail[threadIdx.x] = 0;
}

__global__ void zero_matrix_kernel(unsigned char *c, int rows_bytes, int n, size_t ld_bytes) {
    const int j = blockIdx.y;
    for (int i = blockIdx.x * 256 + threadIdx.x; i < rows_bytes; i += gridDim.x * 256)
        c[(size_t)j * ld_bytes + i] = 0;
}

}  // namespace

// Columns per thread in row mode: kRowChunk, fewer (down to 8) when the
// grid would otherwise hold fewer than ~2048 blocks (small matrices).  Each
// block ends in one atomicMax per row, so longer chunks mean fewer atomics on
// the same addresses (128 rather than 64 columns: the scaling phase of a
// 8192^3 complex call 0.405 -> 0.392 ms).
int row_chunk(int rows, int cols) {
    const long rb = (rows + 255) / 256;
    int chunk = kRowChunk;
    while (chunk > 8 && rb * ((cols + chunk - 1) / chunk) < 2048) chunk >>= 1;
    return chunk;
}

static size_t entry_bytes(ElemType et) { return et == kF64 ? 16 : 8; }

// Non-temporal loads for operands of kStreamBytes and more.
static bool streams(ElemType et, int rows, int cols) {
    return (size_t)rows * (size_t)cols * entry_bytes(et) >= kStreamBytes;
}

template <bool NT>
static void launch_amax_t(int mode, ElemType et, int rows, int cols, const void *X, int ld,
                          unsigned long long *amax, hipStream_t st) {
    if (mode == 0) {
        const int chunk = row_chunk(rows, cols);
        dim3 grid((rows + 255) / 256, (cols + chunk - 1) / chunk);
        switch (et) {
        case kF64: amax_rows<kF64, NT><<<grid, 256, 0, st>>>(rows, cols, chunk, X, ld, amax); break;
        case kF32: amax_rows<kF32, NT><<<grid, 256, 0, st>>>(rows, cols, chunk, X, ld, amax); break;
        case kI32: amax_rows<kI32, NT><<<grid, 256, 0, st>>>(rows, cols, chunk, X, ld, amax); break;
        case kR64: amax_rows<kR64, NT><<<grid, 256, 0, st>>>(rows, cols, chunk, X, ld, amax); break;
        }
    } else {
        dim3 grid(cols, (rows + kColChunk - 1) / kColChunk);
        switch (et) {
        case kF64: amax_cols<kF64, NT><<<grid, 256, 0, st>>>(rows, cols, X, ld, amax); break;
        case kF32: amax_cols<kF32, NT><<<grid, 256, 0, st>>>(rows, cols, X, ld, amax); break;
        case kI32: amax_cols<kI32, NT><<<grid, 256, 0, st>>>(rows, cols, X, ld, amax); break;
        case kR64: amax_cols<kR64, NT><<<grid, 256, 0, st>>>(rows, cols, X, ld, amax); break;
        }
    }
}

hipError_t launch_amax(int mode, ElemType et, int rows, int cols, const void *X, int ld,
                       unsigned long long *amax, hipStream_t st) {
    if (rows <= 0 || cols <= 0) return hipSuccess;
    if (streams(et, rows, cols)) launch_amax_t<true>(mode, et, rows, cols, X, ld, amax, st);
    else launch_amax_t<false>(mode, et, rows, cols, X, ld, amax, st);
    return hipGetLastError();
}

hipError_t launch_exponents(int ca, const unsigned long long *amax_a, int32_t *Ea, int cb,
                            const unsigned long long *amax_b, int32_t *Eb, int *status, hipStream_t st) {
    const int count = ca + cb;
    if (count <= 0) return hipSuccess;
    exponents_kernel<<<(count + 255) / 256, 256, 0, st>>>(ca, amax_a, Ea, cb, amax_b, Eb, status);
    return hipGetLastError();
}

// Columns per thread of the row-mode scan: 32 (a workgroup covers 64 rows x
// 128 columns), fewer (down to 4) when the grid would otherwise hold fewer
// than ~2048 workgroups (small matrices).
int cs_row_cpt(int rows, int cols) {
    const long rb = (rows + 63) / 64;
    int cpt = 32;
    while (cpt > 4 && rb * ((cols + 4 * cpt - 1) / (4 * cpt)) < 2048) cpt >>= 1;
    return cpt;
}

int cs_chunks(int mode, int rows, int cols) {
    if (rows <= 0 || cols <= 0) return 0;
    if (mode == 0) {
        const int w = 4 * cs_row_cpt(rows, cols);
        return (cols + w - 1) / w;
    }
    return (rows + kColChunk - 1) / kColChunk;
}

template <bool NT>
static hipError_t launch_cs_scan_t(int mode, ElemType et, int rows, int cols, const void *X, int ld,
                                   const CsPartials &p, int chunk_ofs, hipStream_t st) {
    if (mode == 0) {
        const int cpt = cs_row_cpt(rows, cols);
        dim3 grid((rows + 63) / 64, (cols + 4 * cpt - 1) / (4 * cpt));
#define O2M_CS_ROWS(T)                                                                                       \
    switch (cpt) {                                                                                           \
    case 32: cs_scan_rows<T, 32, NT><<<grid, 256, 0, st>>>(rows, cols, X, ld, p, chunk_ofs); break;         \
    case 16: cs_scan_rows<T, 16, NT><<<grid, 256, 0, st>>>(rows, cols, X, ld, p, chunk_ofs); break;         \
    case 8: cs_scan_rows<T, 8, NT><<<grid, 256, 0, st>>>(rows, cols, X, ld, p, chunk_ofs); break;           \
    default: cs_scan_rows<T, 4, NT><<<grid, 256, 0, st>>>(rows, cols, X, ld, p, chunk_ofs); break;          \
    }
        switch (et) {
        case kF64: O2M_CS_ROWS(kF64) break;
        case kF32: O2M_CS_ROWS(kF32) break;
        case kR64: O2M_CS_ROWS(kR64) break;
        default: return hipErrorInvalidValue;
        }
#undef O2M_CS_ROWS
    } else {
        if (chunk_ofs != 0) return hipErrorInvalidValue;
        dim3 grid(cols, (rows + kColChunk - 1) / kColChunk);
        switch (et) {
        case kF64: cs_scan_cols<kF64, false, NT><<<grid, 256, 0, st>>>(rows, cols, X, ld, p); break;
        case kF32:
            // chunks start at even rows: an even ld and a 16-byte aligned base align every pair
            if (ld % 2 == 0 && ((uintptr_t)X & 15) == 0)
                cs_scan_cols<kF32, true, NT><<<grid, 256, 0, st>>>(rows, cols, X, ld, p);
            else cs_scan_cols<kF32, false, NT><<<grid, 256, 0, st>>>(rows, cols, X, ld, p);
            break;
        case kR64: cs_scan_cols<kR64, false, NT><<<grid, 256, 0, st>>>(rows, cols, X, ld, p); break;
        default: return hipErrorInvalidValue;
        }
    }
    return hipSuccess;
}

hipError_t launch_cs_scan(int mode, ElemType et, int rows, int cols, const void *X, int ld, const CsPartials &p,
                          int chunk_ofs, hipStream_t st) {
    if (rows <= 0 || cols <= 0) return hipSuccess;
    const hipError_t e = streams(et, rows, cols) ? launch_cs_scan_t<true>(mode, et, rows, cols, X, ld, p, chunk_ofs, st)
                                                 : launch_cs_scan_t<false>(mode, et, rows, cols, X, ld, p, chunk_ofs, st);
    if (e != hipSuccess) return e;
    return hipGetLastError();
}

hipError_t launch_cs_combine(ElemType et, const CsCombineArgs &g, hipStream_t st) {
    const int blocks = (g.ca + 63) / 64 + (g.cb + 63) / 64;
    if (blocks <= 0) return hipSuccess;
    switch (et) {
    case kF64: cs_combine_kernel<kF64><<<blocks, 64 * kCombineWaves, 0, st>>>(g); break;
    case kF32: cs_combine_kernel<kF32><<<blocks, 64 * kCombineWaves, 0, st>>>(g); break;
    case kR64: cs_combine_kernel<kR64><<<blocks, 64 * kCombineWaves, 0, st>>>(g); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_zero(void *p, size_t bytes, hipStream_t st) {
    if (bytes == 0) return hipSuccess;
    const size_t n16 = bytes / 16;
    const int ntail = (int)(bytes % 16);
    size_t blocks = (n16 + 255) / 256;
    if (blocks > 8192) blocks = 8192;
    if (blocks == 0) blocks = 1;
    zero_kernel<<<(unsigned)blocks, 256, 0, st>>>((uint4 *)p, n16, (unsigned char *)p + n16 * 16, ntail);
    return hipGetLastError();
}

hipError_t launch_zero_matrix(void *c, int m, int n, int ldc, int elem_bytes, hipStream_t st) {
    if (m <= 0 || n <= 0) return hipSuccess;
    const int rows_bytes = m * elem_bytes;
    dim3 grid((rows_bytes + 255) / 256 < 64 ? (rows_bytes + 255) / 256 : 64, n);
    zero_matrix_kernel<<<grid, 256, 0, st>>>((unsigned char *)c, rows_bytes, n, (size_t)ldc * elem_bytes);
    return hipGetLastError();
}

}  // namespace o2m
