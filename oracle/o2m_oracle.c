/*
 * CPU oracle for 2M + Ozaki-II complex GEMM.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path links, loads or calls
 * this file; only the test suite, the smoke check and the CPU-baseline leg of
 * the benchmark do.  It shares no code, header, table or constant with the HIP
 * library: every number here is derived from the paper's definitions on its
 * own.
 *
 * Three plain, slow, obviously correct computations:
 *
 *  oracle_gauss_4m  C = AB over Gaussian integers by the classical 4M
 *                   expansion (Section 1), exact in 128-bit integers.  This is
 *                   the result 2M reaches exactly in integer mode (Section 2:
 *                   once the modulus bounds |Re c|, |Im c|, C mod m determines C).
 *
 *  oracle_oq_gemm   The exact output of Algorithm 1 ("2M Ozaki-II"),
 *                   written as its plain definition.  The integer products are
 *                   exact and the CRT + symmetric lift recover the integer
 *                   product C = A_int B_int exactly whenever every |Re c|,
 *                   |Im c| <= (M-1)/2 (Section 3.1), which the scaling budget
 *                   guarantees.  So Algorithm 1 returns
 *                     round(A_int B_int * 2^(E_i + F_j - pA - pB))
 *                   with A_int = round_Z(a * 2^(pA - E_i)) (step 3, componentwise,
 *                   ties to even), computed here in exact multiword integers
 *                   by 4M, and round() one rounding to nearest (ties to even)
 *                   into the output format, fp64 or fp32, subnormals
 *                   included (step 7).  The moduli only enter through pA,
 *                   pB, which the caller derives from M (Python side).
 *
 *  oracle_dd_gemm   The product of the unquantized inputs by 4M in
 *                   double-double (error ~ k 2^-104 |A||B|): the reference the
 *                   accuracy of the method is measured against (Section 6).
 *
 * Matrices are column-major, complex interleaved (re, im), with leading
 * dimensions in complex elements.  Exponent rules (the paper leaves the choice
 * of sigma, tau open, Section 3.1/3.2, pointing to norm- and max-based rules
 * of the Ozaki-II literature):
 *   rule 0 (max):  E_i is the frexp exponent of the largest |Re| or |Im| in
 *                  row i of A (so that max < 2^E_i), 0 for a zero row;
 *   rule 1 (Cauchy-Schwarz): E_i = G with the 2-norm of row i at most 2^G,
 *                  from an exact integer sum of squares (vec_cs_exponent).
 * F_j likewise for column j of B.  A row or column holding Inf or NaN makes
 * its whole row or column of C NaN.
 */
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

typedef __int128 i128;
typedef unsigned __int128 u128;

/* ------------------------------------------------------------------------ */
/* exact integer helpers                                                     */
/* ------------------------------------------------------------------------ */

/* 256-bit two's complement accumulator, little-endian 64-bit words. */
typedef struct { uint64_t w[4]; } acc256;

static void acc_add_shifted(acc256 *a, i128 v, int shift) {
    /* a += v * 2^shift, 0 <= shift < 128 */
    uint64_t x[4];
    int neg = v < 0;
    u128 uv = (u128)v;
    x[0] = (uint64_t)uv;
    x[1] = (uint64_t)(uv >> 64);
    x[2] = x[3] = neg ? ~0ULL : 0ULL;
    while (shift >= 64) {
        x[3] = x[2]; x[2] = x[1]; x[1] = x[0]; x[0] = 0;
        shift -= 64;
    }
    if (shift > 0) {
        x[3] = (x[3] << shift) | (x[2] >> (64 - shift));
        x[2] = (x[2] << shift) | (x[1] >> (64 - shift));
        x[1] = (x[1] << shift) | (x[0] >> (64 - shift));
        x[0] = x[0] << shift;
    }
    unsigned carry = 0;
    for (int t = 0; t < 4; ++t) {
        u128 s = (u128)a->w[t] + x[t] + carry;
        a->w[t] = (uint64_t)s;
        carry = (unsigned)(s >> 64);
    }
}

/* Bit b of the magnitude words w. */
static int bit_of(const uint64_t w[4], int b) { return (int)((w[b >> 6] >> (b & 63)) & 1ULL); }

/* Algorithm 1 step 7 for one component: the exact integer a times 2^scale,
   rounded ONCE to the nearest value of a binary floating-point format with
   `prec` significand bits and least normal exponent emin (fp64: 53, -1022;
   fp32: 24, -126), ties to even, subnormal results included.  Values at or
   beyond the format's largest finite magnitude after rounding become
   infinities (for fp32 when the caller narrows the returned double, which
   holds the rounded value exactly).  A zero integer gives +0; a negative value
   that rounds to zero gives -0. */
static double acc_round(const acc256 *a, int scale, int prec, int emin) {
    uint64_t w[4];
    memcpy(w, a->w, sizeof w);
    int neg = (int64_t)w[3] < 0;
    if (neg) { /* two's complement negate */
        unsigned carry = 1;
        for (int t = 0; t < 4; ++t) {
            u128 s = (u128)(~w[t]) + carry;
            w[t] = (uint64_t)s;
            carry = (unsigned)(s >> 64);
        }
    }
    int top = -1;
    for (int t = 3; t >= 0; --t)
        if (w[t]) { top = 64 * t + 63 - __builtin_clzll(w[t]); break; }
    if (top < 0) return 0.0;
    /* the value lies in [2^e, 2^(e+1)); its quantum (the weight of the last
       significand bit) is 2^(e - prec + 1), but never below the subnormal
       quantum 2^(emin - prec + 1) */
    int e = top + scale;
    int qexp = e - prec + 1;
    if (qexp < emin - prec + 1) qexp = emin - prec + 1;
    int qpos = qexp - scale;                   /* bit of w with weight 2^qexp */
    double r;
    if (qpos <= 0) {
        r = ldexp((double)w[0], scale);        /* fewer than prec bits: exact */
    } else {
        /* significand = bits [qpos, top] (none when qpos > top) */
        uint64_t mant = 0;
        for (int b = top; b >= qpos; --b) mant = (mant << 1) | (uint64_t)bit_of(w, b);
        int round_bit = qpos - 1 <= top ? bit_of(w, qpos - 1) : 0;
        int sticky = 0;
        for (int b = 0; b < qpos - 1 && b <= top; ++b)
            if (bit_of(w, b)) { sticky = 1; break; }
        if (round_bit && (sticky || (mant & 1ULL))) mant += 1; /* may reach 2^prec: still exact */
        r = ldexp((double)mant, qexp);
    }
    return neg ? -r : r;
}

static double acc_to_double(const acc256 *a) { return acc_round(a, 0, 53, -1022); }

static void acc_from_i128(acc256 *a, i128 v) {
    memset(a, 0, sizeof *a);
    acc_add_shifted(a, v, 0);
}

/* ------------------------------------------------------------------------ */
/* scaling exponents                                                         */
/* ------------------------------------------------------------------------ */

/* value x = mant * 2^shift exactly, |mant| <= 2^53, shift >= 0 */
typedef struct { int64_t mant; int shift; } qint;

static qint to_qint(double x) {
    qint q;
    if (fabs(x) < 9007199254740992.0) { /* 2^53: plain integer */
        q.mant = (int64_t)x;
        q.shift = 0;
    } else {
        int e;
        double f = frexp(x, &e);                 /* x = f * 2^e, |f| in [0.5,1) */
        q.mant = (int64_t)ldexp(f, 53);          /* exact: x is an integer with e >= 54 */
        q.shift = e - 53;
    }
    return q;
}

/* Exponent of one complex vector: max over |re|,|im|; returns flag for non-finite. */
static int vec_exponent(const double *x, long stride, int len, int *nonfinite) {
    double amax = 0.0;
    int bad = 0;
    for (int t = 0; t < len; ++t) {
        double re = x[2 * (long)t * stride], im = x[2 * (long)t * stride + 1];
        if (!isfinite(re) || !isfinite(im)) bad = 1;
        double a = fmax(fabs(re), fabs(im));
        if (a > amax) amax = a;
    }
    *nonfinite = bad;
    if (bad || amax == 0.0) return 0;
    int e;
    frexp(amax, &e);
    return e;
}

/* Cauchy-Schwarz exponent of one complex vector x (rule 1).  With E its max
   exponent (vec_exponent), every part v is bounded by u 2^(E-20) with the
   integer u = ceil(|v| 2^(20-E)) <= 2^20 (u = 1 for a nonzero |v| whose
   scaled value underflows: it lies in (0, 1)).  U = sum of u^2 over both
   parts of every entry is exact (below 2^59 for len < 2^17), so
   ||x||_2^2 <= U 4^(E-20).  With d the smallest d >= 0 such that 4^d >= U,
   G = E - 20 + d gives ||x||_2 <= 2^G, and G is at most one above the
   exponent of the norm itself.  A zero vector keeps E = 0. */
static int vec_cs_exponent(const double *x, long stride, int len, int *nonfinite) {
    const int E = vec_exponent(x, stride, len, nonfinite);
    if (*nonfinite) return 0;
    u128 U = 0;
    for (int t = 0; t < len; ++t) {
        for (int part = 0; part < 2; ++part) {
            const double v = x[2 * (long)t * stride + part];
            if (v == 0.0) continue;
            double u = ceil(ldexp(fabs(v), 20 - E));
            if (u < 1.0) u = 1.0;
            U += (u128)((uint64_t)u * (uint64_t)u);
        }
    }
    if (U == 0) return E;
    int d = 0;
    while (((u128)1 << (2 * d)) < U) ++d;
    return E - 20 + d;
}

static int row_exponent(int rule, const double *x, long stride, int len, int *nonfinite) {
    return rule == 1 ? vec_cs_exponent(x, stride, len, nonfinite) : vec_exponent(x, stride, len, nonfinite);
}

/* Quantize one complex entry: round_Z[i] componentwise, RN-even (Algorithm 1, step 3). */
static void quantize(const double *src, int shift, qint *re, qint *im) {
    *re = to_qint(rint(ldexp(src[0], shift)));
    *im = to_qint(rint(ldexp(src[1], shift)));
}

/* ------------------------------------------------------------------------ */
/* O-Z: exact Gaussian-integer 4M                                            */
/* ------------------------------------------------------------------------ */

/* Returns the number of output components that do not fit in int64. */
int oracle_gauss_4m(int m, int n, int k, const int32_t *A, int lda, const int32_t *B, int ldb,
                    int64_t *C, int ldc) {
    int overflow = 0;
#pragma omp parallel for schedule(dynamic) reduction(+ : overflow)
    for (int j = 0; j < n; ++j) {
        for (int i = 0; i < m; ++i) {
            i128 re = 0, im = 0;
            for (int p = 0; p < k; ++p) {
                const int32_t *a = A + 2 * ((long)i + (long)p * lda);
                const int32_t *b = B + 2 * ((long)p + (long)j * ldb);
                /* (ar + i ai)(br + i bi) = (ar br - ai bi) + i (ar bi + ai br) */
                re += (i128)a[0] * b[0] - (i128)a[1] * b[1];
                im += (i128)a[0] * b[1] + (i128)a[1] * b[0];
            }
            if (re > INT64_MAX || re < INT64_MIN) overflow++;
            if (im > INT64_MAX || im < INT64_MIN) overflow++;
            C[2 * ((long)i + (long)j * ldc)] = (int64_t)re;
            C[2 * ((long)i + (long)j * ldc) + 1] = (int64_t)im;
        }
    }
    return overflow;
}

/* ------------------------------------------------------------------------ */
/* O-Q: exact output of Algorithm 1                                          */
/* ------------------------------------------------------------------------ */

/* Exponents of the rows of A (m x k) and columns of B (k x n) under rule
   0 (max) or 1 (Cauchy-Schwarz). */
void oracle_exponents(int m, int n, int k, const double *A, int lda, const double *B, int ldb,
                      int rule, int32_t *E, int32_t *Ebad, int32_t *F, int32_t *Fbad) {
    for (int i = 0; i < m; ++i) {
        int bad;
        E[i] = row_exponent(rule, A + 2 * (long)i, lda, k, &bad);
        Ebad[i] = bad;
    }
    for (int j = 0; j < n; ++j) {
        int bad;
        F[j] = row_exponent(rule, B + 2 * (long)j * ldb, 1, k, &bad);
        Fbad[j] = bad;
    }
}

static void mul_acc(acc256 *acc, i128 *fast, int use_fast, qint x, qint y, int sign) {
    i128 p = (i128)x.mant * (i128)y.mant;
    if (sign < 0) p = -p;
    if (use_fast) *fast += p;
    else acc_add_shifted(acc, p, x.shift + y.shift);
}

/*
 * C (or the listed entries of C) = Algorithm 1 applied to A (m x k), B (k x n)
 * with quantization shifts pA, pB and exponent rule `rule`.  n_entries < 0: the full matrix into C with
 * leading dimension ldc.  n_entries >= 0: entry t = (ei[t], ej[t]) into
 * C[2t], C[2t+1].  out_f32 = 0: C is complex fp64 (double pairs); out_f32 = 1:
 * C is complex fp32 (float pairs), each component the exact scaled integer
 * rounded once to fp32 (CGEMM: never through an fp64 intermediate rounding).
 */
void oracle_oq_gemm(int m, int n, int k, const double *A, int lda, const double *B, int ldb,
                    int pA, int pB, int rule, int out_f32, void *C, int ldc, int n_entries,
                    const int32_t *ei, const int32_t *ej) {
    int32_t *E = (int32_t *)malloc(sizeof(int32_t) * (m > 0 ? m : 1));
    int32_t *Eb = (int32_t *)malloc(sizeof(int32_t) * (m > 0 ? m : 1));
    int32_t *F = (int32_t *)malloc(sizeof(int32_t) * (n > 0 ? n : 1));
    int32_t *Fb = (int32_t *)malloc(sizeof(int32_t) * (n > 0 ? n : 1));
    oracle_exponents(m, n, k, A, lda, B, ldb, rule, E, Eb, F, Fb);

    /* int128 suffices when no quantized value needs a shift (|x| < 2^53: both
       rules keep |x| <= 2^p + sqrt(k/2) < 2^(p+1) <= 2^53 for p <= 52) and
       every partial sum stays below 2^126 (each of the 2k products per
       component is below 2^(pA+pB+2)). */
    int use_fast = pA <= 52 && pB <= 52 && (pA + pB + 3 + (int)ceil(log2((double)k + 1)) < 126);
    long total = n_entries < 0 ? (long)m * n : n_entries;

#pragma omp parallel
    {
        qint *bre = (qint *)malloc(sizeof(qint) * (k > 0 ? k : 1));
        qint *bim = (qint *)malloc(sizeof(qint) * (k > 0 ? k : 1));
        int cached_j = -1;
#pragma omp for schedule(dynamic, 64)
        for (long t = 0; t < total; ++t) {
            int i, j;
            if (n_entries < 0) { j = (int)(t / m); i = (int)(t % m); }
            else { i = ei[t]; j = ej[t]; }
            const long o = n_entries < 0 ? 2 * ((long)i + (long)j * ldc) : 2 * t;
            double *out64 = (double *)C + o;
            float *out32 = (float *)C + o;
            if (Eb[i] || Fb[j]) {
                if (out_f32) { out32[0] = NAN; out32[1] = NAN; }
                else { out64[0] = NAN; out64[1] = NAN; }
                continue;
            }
            if (j != cached_j) {
                for (int p = 0; p < k; ++p)
                    quantize(B + 2 * ((long)p + (long)j * ldb), pB - F[j], &bre[p], &bim[p]);
                cached_j = j;
            }
            acc256 re, im;
            i128 fre = 0, fim = 0;
            memset(&re, 0, sizeof re);
            memset(&im, 0, sizeof im);
            for (int p = 0; p < k; ++p) {
                qint are, aim;
                quantize(A + 2 * ((long)i + (long)p * lda), pA - E[i], &are, &aim);
                /* 4M: Re = ar br - ai bi, Im = ar bi + ai br */
                mul_acc(&re, &fre, use_fast, are, bre[p], +1);
                mul_acc(&re, &fre, use_fast, aim, bim[p], -1);
                mul_acc(&im, &fim, use_fast, are, bim[p], +1);
                mul_acc(&im, &fim, use_fast, aim, bre[p], +1);
            }
            if (use_fast) { acc_from_i128(&re, fre); acc_from_i128(&im, fim); }
            /* step 7: one rounding of c_int 2^(E_i + F_j - pA - pB) */
            int scale = E[i] + F[j] - pA - pB;
            if (out_f32) {
                out32[0] = (float)acc_round(&re, scale, 24, -126);  /* exact narrowing */
                out32[1] = (float)acc_round(&im, scale, 24, -126);
            } else {
                out64[0] = acc_round(&re, scale, 53, -1022);
                out64[1] = acc_round(&im, scale, 53, -1022);
            }
        }
        free(bre);
        free(bim);
    }
    free(E); free(Eb); free(F); free(Fb);
}

/* Exact integer product of the quantized operands, entries only, as 4 signed
   64-bit words per component (little-endian two's complement): for tests that
   compare residues. out has 8 words per entry (re then im). */
void oracle_oq_cint(int m, int n, int k, const double *A, int lda, const double *B, int ldb,
                    int pA, int pB, int rule, int n_entries, const int32_t *ei, const int32_t *ej,
                    uint64_t *out) {
    int32_t *E = (int32_t *)malloc(sizeof(int32_t) * (m > 0 ? m : 1));
    int32_t *Eb = (int32_t *)malloc(sizeof(int32_t) * (m > 0 ? m : 1));
    int32_t *F = (int32_t *)malloc(sizeof(int32_t) * (n > 0 ? n : 1));
    int32_t *Fb = (int32_t *)malloc(sizeof(int32_t) * (n > 0 ? n : 1));
    oracle_exponents(m, n, k, A, lda, B, ldb, rule, E, Eb, F, Fb);
#pragma omp parallel for schedule(dynamic, 16)
    for (long t = 0; t < n_entries; ++t) {
        int i = ei[t], j = ej[t];
        acc256 re, im;
        i128 dummy = 0;
        memset(&re, 0, sizeof re);
        memset(&im, 0, sizeof im);
        for (int p = 0; p < k; ++p) {
            qint are, aim, bre, bim;
            quantize(A + 2 * ((long)i + (long)p * lda), pA - E[i], &are, &aim);
            quantize(B + 2 * ((long)p + (long)j * ldb), pB - F[j], &bre, &bim);
            mul_acc(&re, &dummy, 0, are, bre, +1);
            mul_acc(&re, &dummy, 0, aim, bim, -1);
            mul_acc(&im, &dummy, 0, are, bim, +1);
            mul_acc(&im, &dummy, 0, aim, bre, +1);
        }
        memcpy(out + 8 * t, re.w, 32);
        memcpy(out + 8 * t + 4, im.w, 32);
    }
    free(E); free(Eb); free(F); free(Fb);
}

/* Correct rounding of a signed 128-bit integer given as two words (for pins). */
double oracle_round_i128(uint64_t lo, uint64_t hi) {
    acc256 a;
    i128 v = (i128)(((u128)hi << 64) | lo);
    acc_from_i128(&a, v);
    return acc_to_double(&a);
}

/* The step-7 rounding of a 256-bit signed integer w (little-endian words)
   times 2^scale into fp64 (f32 = 0) or fp32 (f32 = 1), for pins. */
double oracle_round_scaled(const uint64_t *w, int scale, int f32) {
    acc256 a;
    memcpy(a.w, w, sizeof a.w);
    return f32 ? acc_round(&a, scale, 24, -126) : acc_round(&a, scale, 53, -1022);
}

/* ------------------------------------------------------------------------ */
/* O-F: double-double 4M                                                     */
/* ------------------------------------------------------------------------ */

static inline void two_sum(double a, double b, double *s, double *e) {
    double x = a + b, bb = x - a;
    *e = (a - (x - bb)) + (b - bb);
    *s = x;
}

static inline void dd_add_prod(double *hi, double *lo, double a, double b) {
    double p = a * b;
    double pe = fma(a, b, -p);
    double s, e;
    two_sum(*hi, p, &s, &e);
    e += *lo + pe;
    double t = s + e;
    *lo = e - (t - s);
    *hi = t;
}

void oracle_dd_gemm(int m, int n, int k, const double *A, int lda, const double *B, int ldb,
                    double *Chi, double *Clo, int ldc, int n_entries, const int32_t *ei,
                    const int32_t *ej) {
    long total = n_entries < 0 ? (long)m * n : n_entries;
#pragma omp parallel for schedule(dynamic, 64)
    for (long t = 0; t < total; ++t) {
        int i, j;
        long o;
        if (n_entries < 0) { j = (int)(t / m); i = (int)(t % m); o = 2 * ((long)i + (long)j * ldc); }
        else { i = ei[t]; j = ej[t]; o = 2 * t; }
        double rh = 0, rl = 0, ih = 0, il = 0;
        for (int p = 0; p < k; ++p) {
            const double *a = A + 2 * ((long)i + (long)p * lda);
            const double *b = B + 2 * ((long)p + (long)j * ldb);
            dd_add_prod(&rh, &rl, a[0], b[0]);
            dd_add_prod(&rh, &rl, -a[1], b[1]);
            dd_add_prod(&ih, &il, a[0], b[1]);
            dd_add_prod(&ih, &il, a[1], b[0]);
        }
        Chi[o] = rh; Clo[o] = rl;
        Chi[o + 1] = ih; Clo[o + 1] = il;
    }
}

/* Threads an OpenMP parallel region of the oracle uses (for the baseline
   report). */
int oracle_omp_threads(void) { return omp_get_max_threads(); }
