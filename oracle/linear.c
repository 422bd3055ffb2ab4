/* CPU oracle: the plain dense products of the drafting step, in fp64.
 *
 * TEST INFRASTRUCTURE.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg load this library; the GPU path never does.
 *
 * Y[m][n] = sum_k W[n][k] * X[m][k]   (a linear layer without bias, as each
 * fusion FC, projection and the LM head of the drafter is).  W is stored in
 * the model's storage type (bf16 bit patterns or fp32) and is widened to fp64
 * exactly; X and Y are fp64.  One output row of W at a time, every product in
 * fp64.  Nothing else: no blocking, no reduced precision.
 */
#include <stdint.h>
#include <string.h>
#include <stdlib.h>

static inline double bf16_to_f64(uint16_t b) {
  uint32_t u = ((uint32_t)b) << 16;
  float f;
  memcpy(&f, &u, sizeof f);
  return (double)f;
}

void oracle_linear_bf16(const uint16_t *W, const double *X, double *Y,
                        int64_t M, int64_t N, int64_t K) {
#pragma omp parallel
  {
    double *w = (double *)malloc((size_t)K * sizeof(double));
#pragma omp for schedule(static)
    for (int64_t n = 0; n < N; ++n) {
      const uint16_t *row = W + n * K;
      for (int64_t k = 0; k < K; ++k) w[k] = bf16_to_f64(row[k]);
      for (int64_t m = 0; m < M; ++m) {
        const double *x = X + m * K;
        double acc = 0.0;
#pragma omp simd reduction(+ : acc)
        for (int64_t k = 0; k < K; ++k) acc += w[k] * x[k];
        Y[m * N + n] = acc;
      }
    }
    free(w);
  }
}

void oracle_linear_f32(const float *W, const double *X, double *Y,
                       int64_t M, int64_t N, int64_t K) {
#pragma omp parallel
  {
    double *w = (double *)malloc((size_t)K * sizeof(double));
#pragma omp for schedule(static)
    for (int64_t n = 0; n < N; ++n) {
      const float *row = W + n * K;
      for (int64_t k = 0; k < K; ++k) w[k] = (double)row[k];
      for (int64_t m = 0; m < M; ++m) {
        const double *x = X + m * K;
        double acc = 0.0;
#pragma omp simd reduction(+ : acc)
        for (int64_t k = 0; k < K; ++k) acc += w[k] * x[k];
        Y[m * N + n] = acc;
      }
    }
    free(w);
  }
}
