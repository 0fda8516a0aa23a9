// Internal definitions shared by the HIP kernels and the host side of the
// 2M + Ozaki-II library.  Not part of the public C-ABI (include/o2m.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace o2m {

constexpr int kMax2M = 22;        // the 2M moduli (Section 4)
constexpr int kMaxModuli = 32;    // with up to 10 hybrid 3M moduli (Section 3.2)
constexpr int kMaxProducts = 2 * kMax2M + 3 * (kMaxModuli - kMax2M);  // int8 GEMMs per call
constexpr int kMaxLimbs = 6;
constexpr int kMaxDigits = 5;     // base-2^26 digits of a quantized value (K2)
constexpr int kLimbBits = 40;  // CRT limb base 2^40: limb sums stay below 2^53
constexpr int kStatusOverflow = 1;   // device status bit: gauss-mode bound violated
constexpr int kStatusNonfinite = 2;  // device status bit: a row / column held Inf or NaN

// ---------------------------------------------------------------------------
// Operand plane layout (the int8 residue planes A+-, B+- of eq. 2m-pre)
//
// Every operand plane is R_pad x K_pad int8 values, "K-major": the row index
// is a row of A (or a column of B) and k runs inside.  It is stored in the
// order the int8 GEMM consumes it, so that one wave reads one MFMA fragment as
// a single contiguous 1 KB and one thread block copies one pipeline stage as a
// single contiguous 16 KB per operand:
//
//   block of 256 rows x 64 k       = one GEMM stage for one operand (16 KB)
//   fragment of 16 rows x 64 k     = one v_mfma_i32_16x16x64_i8 operand (1 KB)
//   lane chunk of 1 row x 16 k     = the 16 bytes one lane holds
//
// offset(r, kk) = ((rb*KB + kb)*16 + rg)*1024 + lane*16 + (kk & 15)
// with rb = r/256, rg = (r%256)/16, kb = kk/64,
// lane = (r%16) + 16*((kk%64)/16), KB = K_pad/64.
// ---------------------------------------------------------------------------
constexpr int kRowBlock = 256;
constexpr int kStageK = 64;
constexpr int kFragRows = 16;
constexpr int kFragBytes = 1024;
constexpr int kStageBytes = kRowBlock * kStageK;  // 16 KB per operand per stage

__host__ __device__ inline size_t plane_offset(int r, int kk, int kblocks) {
    const int rb = r >> 8, rr = r & 255;
    const int kb = kk >> 6, kr = kk & 63;
    const int rg = rr >> 4;
    const int lane = (rr & 15) + ((kr >> 4) << 4);
    return ((size_t)(rb * kblocks + kb) * 16 + rg) * kFragBytes + lane * 16 + (kr & 15);
}

inline int round_up(int x, int q) { return (x + q - 1) / q * q; }

// ---------------------------------------------------------------------------
// Per-call constants
// ---------------------------------------------------------------------------

// Residue step (eq. 2m-pre): per modulus m, its root s, fl(1/m) and the
// symmetric residues cpow[d-1] of 2^(26 d), d = 1..4, used to reduce a
// quantized integer x = sum_d x_d 2^(26 d) without integer division.  Moduli 0..n2-1 are 2M
// moduli (planes 2l = X+, 2l+1 = X-); moduli n2..n-1 are the 3M extension of a
// hybrid set (planes 2 n2 + 3 (l - n2) + {0, 1, 2} = Xr, Xi, Xr + Xi).
struct ResidueParams {
    int n;                       // number of moduli N
    int n2;                      // of which 2M moduli
    int mod[kMaxModuli];
    int root[kMaxModuli];
    double inv[kMaxModuli];
    double cpow[kMaxModuli][kMaxDigits - 1];
};

// CRT step (eq. 2m-post folded into Algorithm 1 step 5): X_re = sum_l u_l W^re_l,
// X_im = sum_l v_l W^im_l with u = C- + C+, v = C- - C+ and
// W^re_l = (M/m_l) * [((M/m_l)^-1 2^-1) mod m_l],
// W^im_l = (M/m_l) * [((M/m_l)^-1 s_l 2^-1) mod m_l], as T balanced limbs.
// For a 3M modulus of a hybrid set, u = T1 - T2, v = T3 - T1 - T2 (3M post)
// and both parts use the plain weight W_l = (M/m_l) [(M/m_l)^-1 mod m_l],
// stored in wre.
struct CrtParams {
    int n;                        // N
    int n2;                       // 2M moduli among them
    int limbs;                    // T
    double wre[kMaxModuli][kMaxLimbs];
    double wim[kMax2M][kMaxLimbs];
    double mlimb[kMaxLimbs];      // M in balanced limbs
    double inv_m;                 // fl(1/M)
    uint64_t m_lo, m_hi;          // M (gauss mode: M < 2^63, m_hi = 0)
    uint64_t h_lo;                // (M-1)/2 when M < 2^64 (gauss mode)
};

// Host-side tables for one N (built once, cached).
struct ModuliTable {
    int n;
    double log2M;
    ResidueParams res;
    CrtParams crt;
    // exact M as 32-bit words (little endian), for the budget computation
    uint32_t mwords[8];
    int mwords_len;
};

// Returns the table for n moduli (1..kMaxModuli), building it on first use:
// the first min(n, 22) 2M moduli, then n - 22 moduli of the 3M extension.
const ModuliTable *moduli_table(int n);
// The 2M moduli in greedy order (Section 4); returns the count (22).
int moduli_2m(int *out, int cap);
// The hybrid extension (Section 3.2): the greedy scan from 256 down over all
// integers coprime to the 2M set and to each other; returns the count.
int moduli_extension(int *out, int cap);
// Smallest s with s^2 = -1 mod m, or 0 if none.
int root_of_minus_one(int m);
// Largest P with 2k 2^P <= (M-1)/2 - floor(M/2^32).
int budget(const ModuliTable *t, int k);
// Cauchy-Schwarz shifts: the largest S = qA + qB (qA = floor(S/2), qB = S - qA;
// symmetric: qA = qB = floor(S/2)) with (2^qA + R)(2^qB + R) <= (M-1)/2 -
// floor(M/2^32), R = ceil(sqrt(k/2)).  False when no S >= 0 qualifies.
bool budget_cs(const ModuliTable *t, int k, bool symmetric, int *qA, int *qB);

// ---------------------------------------------------------------------------
// Kernel launchers (each .hip file exports its own)
// ---------------------------------------------------------------------------

enum ElemType { kF64 = 0, kF32 = 1, kI32 = 2, kR64 = 3 /* real fp64 */ };

// K1: max |Re|,|Im| per row (mode 0) or per column (mode 1) of a column-major
// matrix, into amax bits (uint64, atomicMax of |x| bit patterns).
hipError_t launch_amax(int mode, ElemType et, int rows, int cols, const void *X, int ld,
                       unsigned long long *amax, hipStream_t st);
// K1 finish: amax bits -> exponents (INT32_MIN when non-finite, which also
// ORs kStatusNonfinite into *status), for ca rows of A and cb columns of B in
// one launch.
hipError_t launch_exponents(int ca, const unsigned long long *amax_a, int32_t *Ea, int cb,
                            const unsigned long long *amax_b, int32_t *Eb, int *status, hipStream_t st);
// K1, Cauchy-Schwarz rule, in one pass over each operand (cs_bounds.h).
// Pass 1 (launch_cs_scan) writes one record per (row, chunk) of row (mode 0)
// or column (mode 1) entries: the chunk's max |Re|,|Im| bit pattern, and the
// sums S2 = sum y^2, S1 = sum y and the count n of nonzero parts, with
// y = max(1, ceil(|v| 2^(20 - e))) against the chunk's own max exponent e.
// Records live at [chunk][entry] with pitch `pitch`; a source's chunks start at
// chunk_ofs (rank-2k rows: A's chunks, then B's).
struct CsPartials {
    unsigned long long *mx, *s2, *s1n;  // s1n = S1 | n << 44
    int pitch;                          // entries per chunk row (padded rows)
    int chunks;                         // chunks per entry, all sources
};
// Chunks per entry that one source of rows x cols gives in `mode`.
int cs_chunks(int mode, int rows, int cols);
hipError_t launch_cs_scan(int mode, ElemType et, int rows, int cols, const void *X, int ld, const CsPartials &p,
                          int chunk_ofs, hipStream_t st);
// Pass 2: E and the Cauchy-Schwarz exponent of every row of A (ca) and column
// of B (cb) from the records (INT32_MIN and kStatusNonfinite for Inf/NaN, 0
// for zero rows); an entry whose records leave the exponent open is summed
// again from the operands (rows: A, and B2 for rank-2k updates; columns: B).
struct CsCombineArgs {
    int ca, cb;
    CsPartials pa, pb;
    int32_t *Ea, *Eb;
    int *status;
    const void *A, *B2, *B;
    int lda, ldb2, ldb;
    int k;                  // entries per row of A (per column of B)
    int amode, bmode;       // how the entries sit in memory: 0 = a row of a
                            // column-major matrix (A's default), 1 = a column
                            // (B's default); B2 (rank-2k) is read as rows
};
hipError_t launch_cs_combine(ElemType et, const CsCombineArgs &g, hipStream_t st);
// K2: quantize + residues + 2M pre into operand planes.
//   mode 0: operand rows are rows of X (A, m x k), element (r, kk) at X[r + kk*ld]
//   mode 1: operand rows are columns of X (B, k x n), element (r, kk) at X[kk + r*ld]
//   mode 2: SYRK, X real n x k, element (r, kk) = X[r + kk*ld] + i X[r + (kk+kh)*ld]
//   shift: quantization shift p (value scaled by 2^(p - E_r)); E may be NULL (gauss).
//   digits: base-2^26 digits of the quantized values, from their bound
//   (residue_digits).
// Plane 2l receives X+ and plane 2l+1 receives X-; the source's k-block j
// lands in k-block j + kofs_p of the + plane and j + kofs_m of the - plane
// (rank-2k updates concatenate two sources along k; otherwise both are 0).
struct PlaneGeom {
    int rows, k;         // logical sizes (SYRK: k = ceil(kreal / 2))
    int kreal;           // SYRK: columns of the real matrix
    int rows_pad, kblocks;   // kblocks: k-blocks of this source
    int plane_kblocks;       // k-blocks of the destination planes
    int kofs_p, kofs_m;      // k-block offsets in the + and - planes
    size_t plane_bytes;  // rows_pad * plane_kblocks * 64
    int conj;            // 1: the operand is conj(X) (a conjugate-transposed GEMM operand)
};
hipError_t launch_residues(int mode, ElemType et, const void *X, int ld, const int32_t *E, int shift,
                           int digits, int khalf, const PlaneGeom &g, const ResidueParams &rp,
                           int8_t *planes, hipStream_t st);
// Digits for quantized values below 2^bits: 1 up to 44 bits (no split), 2 up
// to 62, 3 up to 88 (top digit < 2^36), 4 up to 108 and 5 up to 134 (top digit
// < 2^30, int32); 0 if more are needed.
inline int residue_digits(int bits) {
    return bits <= 44 ? 1 : bits <= 62 ? 2 : bits <= 88 ? 3 : bits <= 108 ? 4 : bits <= 134 ? 5 : 0;
}

// K3: batched int8 GEMM  C_p = A_p B_p^T  (both operands K-major planes), then
// C_p mod m_p stored as int8 (symmetric residue), column-major with leading
// dimension ldc = m_pad, plane stride ldc * n_pad.  mod[p], inv[p]: the
// modulus of product p and its fp64 reciprocal.
// The int8 GEMM's pool counters sit kQueueStride unsigned apart (256 bytes):
// one cache line each, so that claims on different pools do not serialize.
constexpr int kQueueStride = 64;

struct GemmArgs {
    const int8_t *a;
    const int8_t *b;
    int8_t *c;
    size_t a_pstride, b_pstride, c_pstride;  // bytes between consecutive batch items
    int mt, nt, kblocks;                     // tiles along m, n; k stages
    int batch;
    int ldc;
    int chunk;                               // tiles per XCD per product (set by the launcher)
    int deal;                                // 1: 32-tile windows dealt round-robin to the XCDs
    int fixed;                               // slots per XCD taken by workgroup index (launcher)
    unsigned *queue;                         // 8 pool counters, one per XCD, kQueueStride
                                             // apart; zero at launch
    int mod[kMaxProducts];
    double inv[kMaxProducts];
};
hipError_t launch_gemm(const GemmArgs &ga, hipStream_t st);

// K4: CRT + lift + descale.
//   mode 0 ZGEMM  (planes 2l = C+, 2l+1 = C-), output complex
//   mode 1 HERK   (plane l = C+, C- = C+^T), lower triangle, complex
//   mode 2 SYRK   (as HERK, real part only)
//   mode 3 gauss  (as ZGEMM, exact int64 output, status bit on overflow)
//   mode 4 residues hook (as ZGEMM, per-modulus 2M post output)
struct CrtArgs {
    const int8_t *res;
    size_t plane_bytes;
    int ldr;            // leading dimension of residue planes (m_pad)
    int m, n;
    void *c;
    int ldc;
    const int32_t *E, *F;
    int scale_bias;     // -(pA + pB)
    const unsigned long long *amaxA, *amaxB;  // gauss mode bound check
    int k;
    int *status;
    int upper;          // HERK/SYRK/rank-2k: write the upper triangle instead of the lower
    short hmod[kMaxModuli], hroot[kMaxModuli];  // hook mode: moduli and roots
};
// Both go to the CRT kernels by value: stay within the kernel-argument limit.
static_assert(sizeof(CrtArgs) + sizeof(CrtParams) <= 4000, "CRT kernel arguments");
hipError_t launch_crt(int mode, ElemType out_type, const CrtArgs &ca, const CrtParams &cp,
                      hipStream_t st);

// Utility: zero a device buffer with a fill kernel (safe under graph capture).
hipError_t launch_zero(void *p, size_t bytes, hipStream_t st);
// Utility: zero an m x n column-major matrix of elem_bytes elements.
hipError_t launch_zero_matrix(void *c, int m, int n, int ldc, int elem_bytes, hipStream_t st);

}  // namespace o2m
