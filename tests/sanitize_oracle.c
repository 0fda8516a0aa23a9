/* The C oracle's entry points on one input file, for a build with
 * AddressSanitizer and UndefinedBehaviorSanitizer (tests/test_host_sanitizers.py
 * compares the output file with the regular oracle library's results).
 *
 *   argv[1] (input):  int32 m, n, k, pA, pB, rule; complex128 A (m x k) and
 *                     B (k x n), column-major; int32 pairs GA (m x k), GB (k x n)
 *   argv[2] (output): complex128 C (exact Algorithm-1 output), complex64 C32,
 *                     double-double (hi, lo), int64 pairs of the Gaussian 4M
 *                     product, int32 E (m), F (n), and the step-7 rounding of
 *                     c = 2^60 + 2^36 + 1 into fp32 and of v 2^-1122,
 *                     v = 2^90 + 2^47 + 1, into fp64 (doubles)
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

void oracle_oq_gemm(int m, int n, int k, const double *A, int lda, const double *B, int ldb, int pA, int pB,
                    int rule, int out_f32, void *C, int ldc, int n_entries, const int32_t *ei, const int32_t *ej);
void oracle_dd_gemm(int m, int n, int k, const double *A, int lda, const double *B, int ldb, double *Chi,
                    double *Clo, int ldc, int n_entries, const int32_t *ei, const int32_t *ej);
int oracle_gauss_4m(int m, int n, int k, const int32_t *A, int lda, const int32_t *B, int ldb, int64_t *C, int ldc);
void oracle_exponents(int m, int n, int k, const double *A, int lda, const double *B, int ldb, int rule, int32_t *E,
                      int32_t *Ebad, int32_t *F, int32_t *Fbad);
double oracle_round_scaled(const uint64_t *w, int scale, int f32);

static void *xmalloc(size_t bytes) {
    void *p = malloc(bytes ? bytes : 1);
    if (!p) { fprintf(stderr, "out of memory\n"); exit(2); }
    return p;
}

static void rd(void *p, size_t size, size_t count, FILE *f) {
    if (fread(p, size, count, f) != count) { fprintf(stderr, "short input\n"); exit(2); }
}

int main(int argc, char **argv) {
    if (argc != 3) return 2;
    FILE *in = fopen(argv[1], "rb");
    if (!in) return 2;
    int32_t h[6];
    rd(h, sizeof(int32_t), 6, in);
    const int m = h[0], n = h[1], k = h[2], pA = h[3], pB = h[4], rule = h[5];
    double *A = xmalloc(sizeof(double) * 2 * m * k), *B = xmalloc(sizeof(double) * 2 * k * n);
    int32_t *GA = xmalloc(sizeof(int32_t) * 2 * m * k), *GB = xmalloc(sizeof(int32_t) * 2 * k * n);
    rd(A, sizeof(double), (size_t)2 * m * k, in);
    rd(B, sizeof(double), (size_t)2 * k * n, in);
    rd(GA, sizeof(int32_t), (size_t)2 * m * k, in);
    rd(GB, sizeof(int32_t), (size_t)2 * k * n, in);
    fclose(in);

    double *C = xmalloc(sizeof(double) * 2 * m * n), *hi = xmalloc(sizeof(double) * 2 * m * n);
    double *lo = xmalloc(sizeof(double) * 2 * m * n);
    float *C32 = xmalloc(sizeof(float) * 2 * m * n);
    int64_t *G = xmalloc(sizeof(int64_t) * 2 * m * n);
    int32_t *E = xmalloc(sizeof(int32_t) * m), *Eb = xmalloc(sizeof(int32_t) * m);
    int32_t *F = xmalloc(sizeof(int32_t) * n), *Fb = xmalloc(sizeof(int32_t) * n);
    oracle_oq_gemm(m, n, k, A, m, B, k, pA, pB, rule, 0, C, m, -1, NULL, NULL);
    oracle_oq_gemm(m, n, k, A, m, B, k, pA, pB, rule, 1, C32, m, -1, NULL, NULL);
    oracle_dd_gemm(m, n, k, A, m, B, k, hi, lo, m, -1, NULL, NULL);
    if (oracle_gauss_4m(m, n, k, GA, m, GB, k, G, m) != 0) return 3;
    oracle_exponents(m, n, k, A, m, B, k, rule, E, Eb, F, Fb);
    const uint64_t c[4] = {(1ull << 60) + (1ull << 36) + 1, 0, 0, 0};
    const uint64_t v[4] = {(1ull << 47) + 1, 1ull << 26, 0, 0};
    const double r[2] = {oracle_round_scaled(c, 0, 1), oracle_round_scaled(v, -1122, 0)};

    FILE *out = fopen(argv[2], "wb");
    if (!out) return 2;
    fwrite(C, sizeof(double), (size_t)2 * m * n, out);
    fwrite(C32, sizeof(float), (size_t)2 * m * n, out);
    fwrite(hi, sizeof(double), (size_t)2 * m * n, out);
    fwrite(lo, sizeof(double), (size_t)2 * m * n, out);
    fwrite(G, sizeof(int64_t), (size_t)2 * m * n, out);
    fwrite(E, sizeof(int32_t), (size_t)m, out);
    fwrite(F, sizeof(int32_t), (size_t)n, out);
    fwrite(r, sizeof(double), 2, out);
    fclose(out);
    free(A); free(B); free(GA); free(GB); free(C); free(hi); free(lo); free(C32); free(G);
    free(E); free(Eb); free(F); free(Fb);
    return 0;
}
