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
// based rules of the Ozaki-II literature): a second pass bounds the 2-norm of
// every row / column by 2^G with an exact integer sum of squares of the parts
// rounded up to 2^-20 of the row maximum (ssq_*, cs_exponents_kernel).
//
// Bound: HBM.  Algorithmic bytes = the matrix read once per pass (16 B per
// complex fp64 element).  Rows of a column-major A are strided, so a thread owns one
// row and walks a chunk of columns: every load instruction of a wave reads 64
// consecutive rows (1 KB contiguous).  Columns of B are contiguous: a block
// owns a chunk of one column.
#include "o2m_internal.h"

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
template <ElemType ET> struct Raw;
template <> struct Raw<kF64> {
    typedef double2 T;
    static constexpr int n = 2;
    static __device__ inline T load(const void *X, size_t idx) { return reinterpret_cast<const double2 *>(X)[idx]; }
    static __device__ inline T zero() { return make_double2(0.0, 0.0); }
    static __device__ inline unsigned long long bits(T v) { return umax(bits_of(v.x), bits_of(v.y)); }
    static __device__ inline void parts(T v, double (&p)[2]) { p[0] = v.x; p[1] = v.y; }
};
template <> struct Raw<kF32> {
    typedef float2 T;
    static constexpr int n = 2;
    static __device__ inline T load(const void *X, size_t idx) { return reinterpret_cast<const float2 *>(X)[idx]; }
    static __device__ inline T zero() { return make_float2(0.0f, 0.0f); }
    static __device__ inline unsigned long long bits(T v) { return umax(bits_of((double)v.x), bits_of((double)v.y)); }
    static __device__ inline void parts(T v, double (&p)[2]) { p[0] = (double)v.x; p[1] = (double)v.y; }
};
template <> struct Raw<kI32> {
    typedef int2 T;
    static constexpr int n = 2;
    static __device__ inline T load(const void *X, size_t idx) { return reinterpret_cast<const int2 *>(X)[idx]; }
    static __device__ inline T zero() { return make_int2(0, 0); }
    static __device__ inline unsigned long long bits(T v) { return umax(bits_of((double)v.x), bits_of((double)v.y)); }
    static __device__ inline void parts(T v, double (&p)[2]) { p[0] = (double)v.x; p[1] = (double)v.y; }
};
template <> struct Raw<kR64> {
    typedef double T;
    static constexpr int n = 1;
    static __device__ inline T load(const void *X, size_t idx) { return reinterpret_cast<const double *>(X)[idx]; }
    static __device__ inline T zero() { return 0.0; }
    static __device__ inline unsigned long long bits(T v) { return bits_of(v); }
    static __device__ inline void parts(T v, double (&p)[2]) { p[0] = v; p[1] = 0.0; }
};

constexpr int kBatch = 8;   // loads issued together per thread (column mode)

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

constexpr int kRowChunk = 128;    // columns per thread in row mode (at most)
constexpr int kColChunk = 2048;   // rows per block in column mode

template <ElemType ET>
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
    for (int c = c0; c < c1; ++c) best = umax(best, Raw<ET>::bits(Raw<ET>::load(X, (size_t)r + (size_t)c * ld)));
    if (best) atomicMax(amax + r, best);
}

template <ElemType ET>
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
        v[u] = r < r1 ? Raw<ET>::load(X, (size_t)r + (size_t)c * ld) : Raw<ET>::zero();
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

// Cauchy-Schwarz sums of squares (exact in uint64: at most 2 * 2^40 per entry
// and k <= 149130 entries, below 2^59).  Same traversal as the maxima.
template <ElemType ET>
__global__ __launch_bounds__(256) void ssq_rows(int rows, int cols, int chunk, const void *X, int ld,
                                                const int32_t *E, unsigned long long *U) {
    const int r = blockIdx.x * 256 + threadIdx.x;
    if (r >= rows) return;
    const int e = E[r];
    if (e == INT32_MIN) return;
    const int c0 = blockIdx.y * chunk;
    const int c1 = min(cols, c0 + chunk);
    unsigned long long acc = 0;
    auto add = [&](typename Raw<ET>::T x) {
        double v[2];
        Raw<ET>::parts(x, v);
#pragma unroll
        for (int q = 0; q < Raw<ET>::n; ++q) acc += ssq_term(v[q], e);
    };
    for (int c = c0; c < c1; ++c) add(Raw<ET>::load(X, (size_t)r + (size_t)c * ld));
    if (acc) atomicAdd(U + r, acc);
}

template <ElemType ET>
__global__ __launch_bounds__(256) void ssq_cols(int rows, int cols, const void *X, int ld, const int32_t *E,
                                                unsigned long long *U) {
    const int c = blockIdx.x;
    const int e = E[c];
    if (e == INT32_MIN) return;  // uniform over the block
    const int r0 = blockIdx.y * kColChunk;
    const int r1 = min(rows, r0 + kColChunk);
    unsigned long long acc = 0;
    typename Raw<ET>::T x[kBatch];
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
        const int r = r0 + threadIdx.x + 256 * u;
        x[u] = r < r1 ? Raw<ET>::load(X, (size_t)r + (size_t)c * ld) : Raw<ET>::zero();
    }
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
        double v[2];
        Raw<ET>::parts(x[u], v);
#pragma unroll
        for (int q = 0; q < Raw<ET>::n; ++q) acc += ssq_term(v[q], e);
    }
    for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off, 64);
    if ((threadIdx.x & 63) == 0 && acc) atomicAdd(U + c, acc);
}

// E_r -> E_r - 20 + d, d = smallest d >= 0 with 4^d >= U_r, i.e.
// d = ceil(bitlength(U_r - 1) / 2); then ||row r||_2 <= 2^(new E_r).
// Entries [0, ca) of (Ua, Ea), then [0, cb) of (Ub, Eb), in one launch.
__global__ void cs_exponents_kernel(int ca, const unsigned long long *Ua, int32_t *Ea, int cb,
                                    const unsigned long long *Ub, int32_t *Eb) {
    int i = blockIdx.x * 256 + threadIdx.x;
    const unsigned long long *U = Ua;
    int32_t *E = Ea;
    if (i >= ca) { i -= ca; U = Ub; E = Eb; if (i >= cb) return; }
    const int e = E[i];
    const unsigned long long u = U[i];
    if (e == INT32_MIN || u == 0) return;
    const int bits = u == 1 ? 0 : 64 - __clzll((long long)(u - 1));
    E[i] = e - 20 + (bits + 1) / 2;
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

hipError_t launch_amax(int mode, ElemType et, int rows, int cols, const void *X, int ld,
                       unsigned long long *amax, hipStream_t st) {
    if (rows <= 0 || cols <= 0) return hipSuccess;
    if (mode == 0) {
        const int chunk = row_chunk(rows, cols);
        dim3 grid((rows + 255) / 256, (cols + chunk - 1) / chunk);
        switch (et) {
        case kF64: amax_rows<kF64><<<grid, 256, 0, st>>>(rows, cols, chunk, X, ld, amax); break;
        case kF32: amax_rows<kF32><<<grid, 256, 0, st>>>(rows, cols, chunk, X, ld, amax); break;
        case kI32: amax_rows<kI32><<<grid, 256, 0, st>>>(rows, cols, chunk, X, ld, amax); break;
        case kR64: amax_rows<kR64><<<grid, 256, 0, st>>>(rows, cols, chunk, X, ld, amax); break;
        }
    } else {
        dim3 grid(cols, (rows + kColChunk - 1) / kColChunk);
        switch (et) {
        case kF64: amax_cols<kF64><<<grid, 256, 0, st>>>(rows, cols, X, ld, amax); break;
        case kF32: amax_cols<kF32><<<grid, 256, 0, st>>>(rows, cols, X, ld, amax); break;
        case kI32: amax_cols<kI32><<<grid, 256, 0, st>>>(rows, cols, X, ld, amax); break;
        case kR64: amax_cols<kR64><<<grid, 256, 0, st>>>(rows, cols, X, ld, amax); break;
        }
    }
    return hipGetLastError();
}

hipError_t launch_exponents(int ca, const unsigned long long *amax_a, int32_t *Ea, int cb,
                            const unsigned long long *amax_b, int32_t *Eb, int *status, hipStream_t st) {
    const int count = ca + cb;
    if (count <= 0) return hipSuccess;
    exponents_kernel<<<(count + 255) / 256, 256, 0, st>>>(ca, amax_a, Ea, cb, amax_b, Eb, status);
    return hipGetLastError();
}

hipError_t launch_ssq(int mode, ElemType et, int rows, int cols, const void *X, int ld, const int32_t *E,
                      unsigned long long *U, hipStream_t st) {
    if (rows <= 0 || cols <= 0) return hipSuccess;
    if (mode == 0) {
        const int chunk = row_chunk(rows, cols);
        dim3 grid((rows + 255) / 256, (cols + chunk - 1) / chunk);
        switch (et) {
        case kF64: ssq_rows<kF64><<<grid, 256, 0, st>>>(rows, cols, chunk, X, ld, E, U); break;
        case kF32: ssq_rows<kF32><<<grid, 256, 0, st>>>(rows, cols, chunk, X, ld, E, U); break;
        case kR64: ssq_rows<kR64><<<grid, 256, 0, st>>>(rows, cols, chunk, X, ld, E, U); break;
        default: return hipErrorInvalidValue;
        }
    } else {
        dim3 grid(cols, (rows + kColChunk - 1) / kColChunk);
        switch (et) {
        case kF64: ssq_cols<kF64><<<grid, 256, 0, st>>>(rows, cols, X, ld, E, U); break;
        case kF32: ssq_cols<kF32><<<grid, 256, 0, st>>>(rows, cols, X, ld, E, U); break;
        case kR64: ssq_cols<kR64><<<grid, 256, 0, st>>>(rows, cols, X, ld, E, U); break;
        default: return hipErrorInvalidValue;
        }
    }
    return hipGetLastError();
}

hipError_t launch_cs_exponents(int ca, const unsigned long long *Ua, int32_t *Ea, int cb,
                               const unsigned long long *Ub, int32_t *Eb, hipStream_t st) {
    const int count = ca + cb;
    if (count <= 0) return hipSuccess;
    cs_exponents_kernel<<<(count + 255) / 256, 256, 0, st>>>(ca, Ua, Ea, cb, Ub, Eb);
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
