/*
 * Plain FP64 CPU oracle for the W4A16 GEMM of MARLIN (arXiv 2408.11743).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may call, link or
 * load this file: it exists so that the tests and the benchmark's CPU
 * baseline can check the HIP kernels against a slow, obviously correct
 * evaluation of the paper's definition.  It shares no code, header, table
 * or constant with the HIP library.
 *
 * What it computes (Section 3.4, "Kernel Design"): B is a K x N matrix
 * quantised symmetrically to 4 bits, with one fp16 scale per output column
 * or one per run of g consecutive weights of a column, ceil(K/g)*N scales in
 * total.  A code q in 0..15 stands for the signed value q - 8 (Section 3.4,
 * "Dequantization and Tensor Cores": the unsigned 4-bit value is made signed
 * by subtracting 8).  So the weight is
 *
 *     w[k][n] = s[floor(k/g)][n] * (q[k][n] - 8)
 *
 * and the product is the plain matrix product over exactly M*K*N
 * multiply-accumulates (Section 3.4, "Bound By Weight Loading"):
 *
 *     C[m][n] = sum_{k=0}^{K-1} A[m][k] * w[k][n].
 *
 * Arithmetic: A and s are IEEE binary16 inputs widened exactly to double.
 * Each term A*s*(q-8) is exact in double (11 + 11 + 4 significant bits);
 * only the running sum over k (in increasing k) rounds.  The result is not
 * rounded to fp16.
 *
 * The 2:4 variant (Section 4): a pruned position holds weight zero; the
 * oracle takes the dense code matrix with pruned positions already set to
 * code 8, so the same routine covers it.
 *
 * Loops are plain (m, k outer, n inner); OpenMP splits the n range only,
 * which leaves every summation order unchanged.
 */
#include <math.h>
#include <stddef.h>
#include <stdint.h>
#include <stdlib.h>

/* IEEE 754 binary16 -> double, from the format's definition: 1 sign bit,
 * 5 exponent bits (bias 15), 10 fraction bits; exponent 0 encodes zero and
 * subnormals (fraction * 2^-24), exponent 31 encodes infinities and NaNs. */
double oracle_f16_to_f64(uint16_t h)
{
    int sign = (h >> 15) & 1;
    int e = (h >> 10) & 0x1f;
    int f = h & 0x3ff;
    double v;
    if (e == 0) {
        v = ldexp((double)f, -24);
    } else if (e == 31) {
        v = (f == 0) ? INFINITY : NAN;
    } else {
        v = ldexp((double)(1024 + f), e - 25);
    }
    return sign ? -v : v;
}

/* Scale row that covers row k of B: floor(k / g); g == K (or g <= 0) means
 * one scale row for the whole column. */
static int64_t scale_row(int64_t k, int64_t K, int64_t g)
{
    if (g <= 0 || g >= K) return 0;
    return k / g;
}

/* w[k][n] = s[floor(k/g)][n] * (q[k][n] - 8), written out as double.
 * q: uint8 [K][N], low nibble is the code.  s: fp16 bits [ceil(K/g)][N]. */
void oracle_dequant(const uint8_t *q, const uint16_t *s, int64_t K, int64_t N,
                    int64_t g, double *w)
{
    for (int64_t k = 0; k < K; ++k) {
        const int64_t r = scale_row(k, K, g);
        for (int64_t n = 0; n < N; ++n) {
            const int code = q[k * N + n] & 0xf;
            w[k * N + n] = oracle_f16_to_f64(s[r * N + n]) * (double)(code - 8);
        }
    }
}

/* Widen n fp16 values to double with oracle_f16_to_f64. */
static double *widen(const uint16_t *h, int64_t n)
{
    double *d = (double *)malloc((size_t)(n > 0 ? n : 1) * sizeof(double));
    if (!d) abort();
    for (int64_t i = 0; i < n; ++i) d[i] = oracle_f16_to_f64(h[i]);
    return d;
}

/* C[m][n] = sum_k A[m][k] * s[floor(k/g)][n] * (q[k][n] - 8), in double.
 * A: fp16 bits [M][K].  q: uint8 [K][N].  s: fp16 bits [ceil(K/g)][N].
 * C: double [M][N], overwritten.  A and s are widened to double once up
 * front; that changes no value (the widening is exact). */
void oracle_gemm(const uint16_t *A, const uint8_t *q, const uint16_t *s,
                 int64_t M, int64_t N, int64_t K, int64_t g, double *C)
{
    const int64_t G = (g <= 0 || g >= K) ? 1 : (K + g - 1) / g;
    double *Ad = widen(A, M * K);
    double *sd = widen(s, G * N);
    const int64_t NB = 256; /* columns per parallel chunk */
    const int64_t nchunks = (N + NB - 1) / NB;
#pragma omp parallel for schedule(dynamic)
    for (int64_t c = 0; c < nchunks; ++c) {
        const int64_t n0 = c * NB;
        const int64_t n1 = (n0 + NB < N) ? n0 + NB : N;
        for (int64_t m = 0; m < M; ++m) {
            double *crow = C + m * N;
            for (int64_t n = n0; n < n1; ++n) crow[n] = 0.0;
            for (int64_t k = 0; k < K; ++k) {
                const double a = Ad[m * K + k];
                const uint8_t *qrow = q + k * N;
                const double *srow = sd + scale_row(k, K, g) * N;
                for (int64_t n = n0; n < n1; ++n) {
                    const double w = srow[n] * (double)((qrow[n] & 0xf) - 8);
                    crow[n] += a * w;
                }
            }
        }
    }
    free(Ad);
    free(sd);
}

/* The same sum for a list of single outputs (m_idx[i], n_idx[i]); used where
 * the full product is too large for the CPU.  out: double [count]. */
void oracle_gemm_sampled(const uint16_t *A, const uint8_t *q, const uint16_t *s,
                         int64_t M, int64_t N, int64_t K, int64_t g,
                         const int64_t *m_idx, const int64_t *n_idx, int64_t count,
                         double *out)
{
    (void)M;
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < count; ++i) {
        const int64_t m = m_idx[i], n = n_idx[i];
        double acc = 0.0;
        for (int64_t k = 0; k < K; ++k) {
            const double a = oracle_f16_to_f64(A[m * K + k]);
            const double w = oracle_f16_to_f64(s[scale_row(k, K, g) * N + n]) *
                             (double)((q[k * N + n] & 0xf) - 8);
            acc += a * w;
        }
        out[i] = acc;
    }
}
