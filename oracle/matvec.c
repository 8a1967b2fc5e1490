/* Plain float64 matrix-vector products over stored weights.
 *
 * TEST INFRASTRUCTURE ONLY: part of the float64 oracle.  Nothing on the product
 * path links or calls this file.  It lets the oracle run a long greedy decode of
 * a full-size model without widening every weight matrix to float64 on each step.
 * It computes the same products as a float64 matrix multiply of the widened
 * weights; only the order of the additions differs.
 *
 *   Y[t][n] = sum_k W[n][k] * X[t][k]        t < T, n < N, k < K
 *
 * W is row-major [N][K], stored either as bfloat16 bit patterns (the upper 16
 * bits of a float32) or as float32 values.  X [T][K] and Y [T][N] are float64.
 * Every weight is widened exactly to float64.  Each product and sum is a float64
 * operation.  The sum over k is formed as eight partial sums, where partial r
 * takes k = r, r + 8, r + 16, ... in increasing order, and the eight are then
 * added in index order.  Rows are shared among OpenMP threads.  No thread
 * writes another thread's rows, so the result does not depend on the thread
 * count.
 */

#include <stdint.h>
#include <string.h>

static inline double widen_bf16(uint16_t b)
{
    uint32_t u = (uint32_t)b << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

#define DOT_BODY(LOAD)                                                        \
    double p[8] = {0, 0, 0, 0, 0, 0, 0, 0};                                   \
    int64_t k = 0;                                                            \
    for (; k + 8 <= K; k += 8)                                                \
        for (int r = 0; r < 8; ++r) p[r] += LOAD(w[k + r]) * x[k + r];        \
    for (int r = 0; k < K; ++k, ++r) p[r] += LOAD(w[k]) * x[k];              \
    double s = 0.0;                                                           \
    for (int r = 0; r < 8; ++r) s += p[r];                                    \
    return s;

static inline double widen_f32(float v) { return (double)v; }

static double dot_bf16(const uint16_t* w, const double* x, int64_t K) { DOT_BODY(widen_bf16) }
static double dot_f32(const float* w, const double* x, int64_t K) { DOT_BODY(widen_f32) }

/* Returns 0 on success, -1 on a bad size. */
int oracle_matvec_bf16(const uint16_t* W, int64_t N, int64_t K, const double* X, int64_t T,
                       double* Y)
{
    if (N < 0 || K < 0 || T < 0) return -1;
#pragma omp parallel for schedule(static)
    for (int64_t n = 0; n < N; ++n)
        for (int64_t t = 0; t < T; ++t)
            Y[t * N + n] = dot_bf16(W + n * K, X + t * K, K);
    return 0;
}

int oracle_matvec_f32(const float* W, int64_t N, int64_t K, const double* X, int64_t T,
                      double* Y)
{
    if (N < 0 || K < 0 || T < 0) return -1;
#pragma omp parallel for schedule(static)
    for (int64_t n = 0; n < N; ++n)
        for (int64_t t = 0; t < T; ++t)
            Y[t * N + n] = dot_f32(W + n * K, X + t * K, K);
    return 0;
}
