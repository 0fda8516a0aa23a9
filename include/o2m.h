/*
 * o2m.h -- complex GEMM, HERK and SYRK by 2M multiplication combined with the
 * Ozaki-II scheme, on int8 matrix cores of AMD Instinct MI355X (gfx950).
 *
 * Method: "The 2M Multiplication Algorithm for Complex Matrices" (Caday).
 *   Section 2     2M multiplication: for an odd modulus m with s^2 = -1 (mod m)
 *                 a complex product of integer matrices modulo m costs two real
 *                 products, C+ = A+ B+ and C- = A- B- with A+- = Ar +- s Ai.
 *   Section 3.2   Algorithm 1 ("2M Ozaki-II"): scale rows of A and columns of
 *                 B by powers of two, quantize to Gaussian integers, run 2M
 *                 modulo each of N coprime 2M moduli <= 256 (int8 GEMMs), and
 *                 recover the exact integer product by the Chinese remainder
 *                 theorem with a symmetric lift, then undo the scaling.
 *   Section 4     The 2M moduli: the greedy set {241, 233, 229, 221, 205, ...,
 *                 37, 29} (22 moduli, product ~2^152); N = 16 gives ~2^117.
 *   Section 5     HERK: C- = C+^T, so one int8 GEMM per modulus; SYRK: A A^T
 *                 = Re(Z Z^H) with Z = A1 + i A2 (half the k); HER2K with a
 *                 shared row scale: C+ = A+ B-^T + B+ A-^T is one GEMM over
 *                 [A+ | B+] and [B- | A-]; SYR2K = the half-k HER2K.
 *
 * Conventions for every call below
 *   - Matrices are column-major.  Complex matrices are interleaved (re, im);
 *     leading dimensions count complex elements.  alpha = 1, beta = 0 (the
 *     setting of the paper's experiments, Section 6).
 *   - A, B, C are DEVICE pointers owned by the caller; the library never frees
 *     or retains them.  C must not overlap A or B.
 *   - stream is a hipStream_t (NULL = the default stream).  Calls enqueue
 *     their kernels on it and return without synchronizing; the output is
 *     ready when the stream reaches that point.
 *   - n_moduli is N, the number of moduli used; accuracy grows by about 3.7
 *     bits per modulus and int8 GEMM work grows linearly in N.  N <= 22 uses
 *     the 2M moduli only.  The GEMM calls (zgemm, cgemm, the residue hook)
 *     accept N up to 32: a hybrid set (Section 3.2) where moduli 23..N are the
 *     greedy continuation over all integers <= 256 coprime to the set
 *     (256, 253, 251, 249, 239, 227, 223, 217, 211, 199), none a 2M modulus,
 *     each multiplied with 3M (three int8 GEMMs: Ar Br, Ai Bi,
 *     (Ar + Ai)(Br + Bi) mod m).  Residues mod 256 reach 128, so hybrid sets
 *     need k <= 131071.  HERK/SYRK/rank-2k calls take N <= 22.
 *   - Scaling rules (Algorithm 1 step 2; the paper leaves the choice of the
 *     power-of-two scales open).  k below is the inner dimension of the int8
 *     GEMMs: k for GEMM/HERK, ceil(k/2) for SYRK, twice those for the rank-2k
 *     updates.
 *     O2M_SCALE_MAX (the plain calls): E_i = frexp exponent of the largest
 *       |Re| or |Im| in row i of A (F_j: column j of B); P = the largest
 *       integer with 2k 2^P <= (M-1)/2 - floor(M/2^32); pA = floor(P/2),
 *       pB = P - pA (symmetric ops: pA = pB = floor(P/2)).
 *     O2M_SCALE_CS (the _ex calls): E_i = the smallest G with ||row i||_2 <=
 *       2^G as certified by U = sum over all parts v of ceil(|v| 2^(20-e))^2
 *       (e: the max-rule exponent of the row), i.e. E_i = e - 20 +
 *       ceil(log4 U); (pA, pB) = the largest pA + pB (split as above) with
 *       (2^pA + R)(2^pB + R) <= (M-1)/2 - floor(M/2^32), R = ceil(sqrt(k/2)):
 *       by the Cauchy-Schwarz inequality every |Re c|, |Im c| then stays
 *       recoverable.  Rows with a few dominant entries keep more bits than
 *       under the max rule.
 *     Entries are quantized as rint(a 2^(pA - E_i)), ties to even.  Each
 *     output component equals the exact integer product of the quantized
 *     operands times 2^(E_i + F_j - pA - pB), rounded ONCE to nearest (ties
 *     to even) into the output type: fp64, or fp32 for CGEMM (never through
 *     an fp64 rounding first), subnormal results included (Algorithm 1,
 *     step 7).
 *   - Rows of A or columns of B containing Inf or NaN give NaN in the
 *     corresponding rows / columns of C; zero rows or columns give +0.
 *   - m == 0 or n == 0: nothing is done.  k == 0: C is set to zero.
 *
 * Workspace: the library needs device scratch memory for the residue planes
 * (size: o2m_workspace_bytes).  Each stream of each device has its own: calls
 * on one stream run in order and share it, calls on different streams never
 * share scratch memory, so they may overlap in time.  The library allocates a
 * stream's workspace on its first call and grows it as needed (hipMalloc,
 * after synchronizing that stream); o2m_release_workspace frees it.  A caller
 * may instead bind its own buffer to a stream with o2m_set_workspace.  A
 * workspace is keyed by the stream handle: a stream destroyed while its calls
 * still run must not be replaced by a new stream with the same handle before
 * they finish.
 *
 * Graph capture: once the workspace of the capturing stream is large enough
 * for a call (an earlier call of the same or a larger size on that stream, or
 * o2m_set_workspace for it), the call enqueues kernels only (no allocation,
 * no host synchronisation, no memset: buffers are cleared by kernels), so it
 * can be captured into a HIP graph on its stream and replayed; each replay
 * reads the captured input buffers anew.  A call under capture that would
 * need a larger workspace fails with O2M_ERR_WORKSPACE and leaves the capture
 * intact.  With phase timing on, the captured call records its events as
 * well.
 *
 * Return value: O2M_OK, or a negative code.  -1 .. -12: the position of the
 * first invalid argument (BLAS convention, counting from 1).  Errors found
 * before anything is enqueued leave C untouched.
 */
#ifndef O2M_H
#define O2M_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int o2m_status;

#define O2M_OK 0
#define O2M_ERR_NMODULI (-20)   /* n_moduli outside 1..32 (GEMM), 1..22 (symmetric
                                   calls), 1..8 (gauss mode)                        */
#define O2M_ERR_KLIMIT (-21)    /* k > 149130 (131071 when N > 22): int32
                                   accumulation could overflow                      */
#define O2M_ERR_WORKSPACE (-22) /* workspace too small: a caller buffer, or a stream
                                   under graph capture whose workspace was not
                                   sized before the capture                        */
#define O2M_ERR_HIP (-23)       /* a HIP runtime call or kernel launch failed       */
#define O2M_ERR_NOMEM (-24)     /* workspace allocation failed                      */
#define O2M_ERR_SIZE (-25)      /* a padded size or plane offset exceeds the range  */
#define O2M_ERR_SCALING (-26)   /* unknown scaling rule, or the Cauchy-Schwarz rule
                                   has no valid shifts for this n_moduli and k      */
#define O2M_ERR_SCRATCH (-27)   /* zgemm_2m_noalloc: the call needs more than
                                   O2M_NOALLOC_SCRATCH_BYTES of scratch memory      */

/* scaling rules for the _ex calls */
#define O2M_SCALE_MAX 0         /* max rule (what the plain calls use)              */
#define O2M_SCALE_CS 1          /* Cauchy-Schwarz (2-norm) rule                     */

/* device status bits, read with o2m_get_status */
#define O2M_STATUS_OVERFLOW 1   /* gauss mode: 2k max|A_i| max|B_j| > (M-1)/2    */
#define O2M_STATUS_NONFINITE 2  /* a row of A or column of B held Inf or NaN (its
                                   row / column of C is NaN); Algorithm 1 is
                                   silent on non-finite inputs                    */

#define O2M_MAX_MODULI 22          /* 2M moduli (Section 4)                        */
#define O2M_MAX_MODULI_HYBRID 32   /* GEMM calls with the 3M extension (Section 3.2) */
#define O2M_MAX_K 149130
#define O2M_MAX_K_HYBRID 131071    /* k limit once N > 22 (residues mod 256)         */

/* C = A B, A m x k, B k x n, complex128 (Section 3.2, Algorithm 1). */
o2m_status zgemm_2m(int m, int n, int k, const double *A, int lda, const double *B, int ldb,
                    double *C, int ldc, int n_moduli, void *stream);

/* zgemm_2m_ex for callers that cannot allocate device memory (code under HIP
   graph capture, tight serving loops, harnesses that forbid hipMalloc): the
   same computation and result, with every scratch buffer in a static device
   array of O2M_NOALLOC_SCRATCH_BYTES (256 MiB) that is part of the library's
   device code: every GPU the library's code is loaded on holds a copy until
   the process ends, whether or not this call is used.  The call
   allocates nothing (no hipMalloc, hipFree or allocating library routine),
   enqueues kernels only and returns O2M_ERR_SCRATCH, before anything is
   enqueued, when the call needs more (o2m_workspace_bytes('z', ...) >
   O2M_NOALLOC_SCRATCH_BYTES; e.g. m = n = k = 1024 at N = 16 fits, 2048^3
   does not).  The caller passes A, B and C.  All zgemm_2m_noalloc calls on
   one GPU share its array: calls that overlap in time on one GPU (on
   different streams, or from several threads) race and give wrong results. */
#define O2M_NOALLOC_SCRATCH_BYTES (256u << 20)
o2m_status zgemm_2m_noalloc(int m, int n, int k, const double *A, int lda, const double *B, int ldb,
                            double *C, int ldc, int n_moduli, int scaling, void *stream);

/* C = A B in complex64: fp32 inputs are widened exactly, the same algorithm
   runs, and the result is rounded once to fp32 (Section 3.2; accuracy near fp32
   needs about 8 moduli). */
o2m_status cgemm_2m(int m, int n, int k, const float *A, int lda, const float *B, int ldb,
                    float *C, int ldc, int n_moduli, void *stream);

/* HERK, C = A A^H, A n x k complex128 (Section 5): one int8 GEMM per modulus
   (C+ = A+ A-^T, C- = C+^T).  uplo 'L' or 'l': the lower triangle including
   the diagonal is written, with Im(c_ii) = 0 exactly, and the strictly upper
   triangle of C is not touched; 'U' or 'u': the upper triangle likewise (the
   Section 5 text allows either; both are the same exact values, c_ji =
   conj(c_ij)). */
o2m_status zherk_2m(char uplo, int n, int k, const double *A, int lda, double *C, int ldc,
                    int n_moduli, void *stream);

/* SYRK, C = A A^T, A n x k real fp64 (Section 5): Z = A[:, :k'] + i A[:, k':]
   with k' = ceil(k/2) (a zero column pads odd k), C = Re(Z Z^H) by the 2M
   HERK.  uplo 'L' or 'l' ('U' or 'u'): lower (upper) triangle of the real
   n x n C written. */
o2m_status dsyrk_2m(char uplo, int n, int k, const double *A, int lda, double *C, int ldc,
                    int n_moduli, void *stream);

/* HER2K, C = A B^H + B A^H, A and B n x k complex128 (Section 5).  Row i of
   A and row i of B share one scale (sigma = tau), so the two products add in
   the residue domain: per modulus one int8 GEMM over k' = 2k,
   C+ = [A+ | B+] [B- | A-]^T, and C- = C+^T.  uplo 'L' or 'l' ('U' or 'u'):
   the lower (upper) triangle with Im(c_ii) = 0 exactly is written.  Requires
   2k <= 149130. */
o2m_status zher2k_2m(char uplo, int n, int k, const double *A, int lda, const double *B, int ldb,
                     double *C, int ldc, int n_moduli, void *stream);

/* SYR2K, C = A B^T + B A^T, A and B n x k real fp64 (Section 5): the HER2K of
   Z_A = A[:, :k'] + i A[:, k':] and Z_B likewise, k' = ceil(k/2), real part.
   uplo 'L' or 'l' ('U' or 'u'): lower (upper) triangle.  Requires
   2 ceil(k/2) <= 149130. */
o2m_status dsyr2k_2m(char uplo, int n, int k, const double *A, int lda, const double *B, int ldb,
                     double *C, int ldc, int n_moduli, void *stream);

/* The calls above with an explicit scaling rule (O2M_SCALE_MAX or
   O2M_SCALE_CS, see the conventions).  Same arguments otherwise. */
o2m_status zgemm_2m_ex(int m, int n, int k, const double *A, int lda, const double *B, int ldb,
                       double *C, int ldc, int n_moduli, int scaling, void *stream);
o2m_status cgemm_2m_ex(int m, int n, int k, const float *A, int lda, const float *B, int ldb,
                       float *C, int ldc, int n_moduli, int scaling, void *stream);
o2m_status zherk_2m_ex(char uplo, int n, int k, const double *A, int lda, double *C, int ldc,
                       int n_moduli, int scaling, void *stream);
o2m_status dsyrk_2m_ex(char uplo, int n, int k, const double *A, int lda, double *C, int ldc,
                       int n_moduli, int scaling, void *stream);
o2m_status zher2k_2m_ex(char uplo, int n, int k, const double *A, int lda, const double *B, int ldb,
                        double *C, int ldc, int n_moduli, int scaling, void *stream);
o2m_status dsyr2k_2m_ex(char uplo, int n, int k, const double *A, int lda, const double *B, int ldb,
                        double *C, int ldc, int n_moduli, int scaling, void *stream);

/* C = op(A) op(B) (Section 3.2, Algorithm 1, on the operands op(A), op(B)),
   with op(X) = X for 'N', X^T for 'T' and X^H for 'C' (either case), BLAS
   style: op(A) is m x k, stored as A (m x k, lda >= m) for 'N' or as an
   k x m matrix (lda >= k) otherwise; op(B) is k x n, stored k x n (ldb >= k)
   for 'N' or n x k (ldb >= n) otherwise.  Transposition and conjugation are
   exact and no operand is copied: the kernels read rows of op(A) as columns
   of the stored A when transposed, and conjugation negates imaginary parts as
   they are read (it exchanges A+ and A- of eq. 2m-pre).  The result is that
   of zgemm_2m_ex / cgemm_2m_ex on the explicitly formed op(A), op(B), bit for
   bit.  Argument errors: -1 transa, -2 transb, -3 m, -4 n, -5 k, -6 A,
   -7 lda, -8 B, -9 ldb, -10 C, -11 ldc. */
o2m_status zgemm_2m_op(char transa, char transb, int m, int n, int k, const double *A, int lda,
                       const double *B, int ldb, double *C, int ldc, int n_moduli, int scaling,
                       void *stream);
o2m_status cgemm_2m_op(char transa, char transb, int m, int n, int k, const float *A, int lda,
                       const float *B, int ldb, float *C, int ldc, int n_moduli, int scaling,
                       void *stream);

/* Exact Gaussian-integer product (Section 2): A m x k and B k x n with int32
   (re, im) pairs, C m x n with int64 (re, im) pairs.  No scaling: 2M modulo
   N moduli with N <= 8 (M < 2^63).  Exact when every entry satisfies
   2k max_p|A_ip| max_p|B_pj| <= (M-1)/2 (max over Re and Im parts);
   otherwise the device status bit O2M_STATUS_OVERFLOW is set. */
o2m_status gauss_gemm_2m(int m, int n, int k, const int32_t *A, int lda, const int32_t *B,
                         int ldb, int64_t *C, int ldc, int n_moduli, void *stream);

/* Test hook for zgemm_2m: the per-modulus result of the 2M post step
   (eq. 2m-post), i.e. (Re c_ij mod m_l, Im c_ij mod m_l) of the exact
   quantized product, in the symmetric range [-(m_l-1)/2, (m_l-1)/2].
   res is a device int8 array [n_moduli][2][n][m] (column-major m x n planes,
   Re plane then Im plane per modulus; for the 3M moduli of a hybrid set the
   3M post step, Re = T1 - T2, Im = T3 - T1 - T2); E, F (device int32, may be NULL)
   receive the row / column exponents, with INT32_MIN for a non-finite row /
   column. */
o2m_status zgemm_2m_residues(int m, int n, int k, const double *A, int lda, const double *B,
                             int ldb, int n_moduli, int8_t *res, int32_t *E, int32_t *F,
                             void *stream);
/* The same with an explicit scaling rule; E, F then hold that rule's exponents. */
o2m_status zgemm_2m_residues_ex(int m, int n, int k, const double *A, int lda, const double *B,
                                int ldb, int n_moduli, int scaling, int8_t *res, int32_t *E,
                                int32_t *F, void *stream);

/* Host-only: the first n_moduli moduli (1..32: the 2M moduli of Section 4,
   then the hybrid 3M extension), the smallest square roots of -1 of the 2M
   ones (Section 2; 0 for the 3M ones) and log2 of their product.  Any
   pointer may be NULL.  Touches no GPU. */
o2m_status o2m_moduli(int n_moduli, int32_t *m_out, int32_t *s_out, double *log2M_out);

/* Host-only: the budget P of the max rule for a given n_moduli and inner
   dimension k of the int8 GEMMs. */
o2m_status o2m_budget(int n_moduli, int k, int *P_out);

/* Host-only: the quantization shifts (pA, pB) a call uses.  op as for
   o2m_workspace_bytes, k the call's own k (the SYRK split and the rank-2k
   doubling are applied here).  Returns O2M_ERR_SCALING when the rule has no
   valid shifts (the call would fail the same way). */
o2m_status o2m_shifts(char op, int n_moduli, int k, int scaling, int *pA_out, int *pB_out);

/* Bytes of workspace a call needs.  op: 'z' zgemm, 'c' cgemm, 'h' zherk,
   's' dsyrk, 'x' zher2k, 'y' dsyr2k, 'g' gauss, 'r' zgemm_2m_residues.
   Touches no GPU. */
size_t o2m_workspace_bytes(char op, int m, int n, int k, int n_moduli);

/* Use caller-owned device memory (on the current device) as the workspace of
   the calls on `stream` from now on; NULL returns that stream to
   library-managed memory.  The caller keeps ownership and must keep the
   buffer alive while calls using it may still run.  Calls whose workspace
   exceeds `bytes` fail with O2M_ERR_WORKSPACE. */
o2m_status o2m_set_workspace(void *dev_ptr, size_t bytes, void *stream);

/* Free the library-owned workspace of `stream` on the current device, after
   synchronizing that stream (the next call on it allocates anew). */
o2m_status o2m_release_workspace(void *stream);

/* Synchronize stream, return the device status bits of the current device in
   *device_status and clear them.  The bits are shared by the device's
   streams: they are the OR over every call since the last read. */
o2m_status o2m_get_status(void *stream, int *device_status);

/* Phase timing for profiling: when enabled (which also restarts the count),
   every call records HIP events around its phases (scale, residues, int8 GEMM,
   CRT) on its stream, for up to 1024 calls.  o2m_phase_times waits for the
   last timed call's events and writes, for up to max_phases phases, the
   average elapsed milliseconds over the calls timed since enabling; it returns
   the number of phases written (0 if no call was timed) or -1 on a HIP error
   (for instance when a timed call on another thread has not yet recorded its
   events).  Calls from several threads take separate event slots. */
o2m_status o2m_phase_timing(int enable);
int o2m_phase_times(float *ms, int max_phases);

/* Human-readable text for a status code. */
const char *o2m_status_string(o2m_status status);

#ifdef __cplusplus
}
#endif

#endif /* O2M_H */
