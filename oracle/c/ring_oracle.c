/*
 * Oracle (test infrastructure and the CPU baseline): plain C loops over all
 * host cores (OpenMP over output rows), written from the definitions.
 *
 * oracle_ring_matmul_nt: C = A B^T over Z_{2^32} (the ring of Section 6.1,
 *   k = 32): C[i][j] = sum_t A[i][t] B[j][t] mod 2^32. Unsigned 32-bit
 *   multiply and add wrap around modulo 2^32 in C, so the loop is the
 *   definition itself. A is m x k (leading dimension lda), B is n x k (ldb),
 *   C is m x n (ldc), all row-major uint32.
 *
 * oracle_rotate_rows: the random Hadamard rotation of Section 5 on every
 *   row of x (rows x n, float64, in place): forward y = H (d * v) / sqrt(n),
 *   inverse y = d * (H v) / sqrt(n), with H the Sylvester-ordered
 *   Walsh-Hadamard matrix applied by Fino's butterflies (a, b) ->
 *   (a + b, a - b) over log2(n) stages; n a power of two; d (signs, +-1,
 *   NULL for none).
 */
#include <math.h>
#include <omp.h>
#include <stdint.h>

void oracle_ring_matmul_nt(const uint32_t* A, int64_t lda, const uint32_t* B, int64_t ldb, uint32_t* C,
                           int64_t ldc, int64_t m, int64_t n, int64_t k) {
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t i = 0; i < m; ++i) {
    const uint32_t* a = A + i * lda;
    for (int64_t j = 0; j < n; ++j) {
      const uint32_t* b = B + j * ldb;
      uint32_t s = 0;
      for (int64_t t = 0; t < k; ++t) s += a[t] * b[t];
      C[i * ldc + j] = s;
    }
  }
}

void oracle_rotate_rows(double* x, int64_t rows, int64_t n, const int8_t* signs, int inverse) {
  const double scale = 1.0 / sqrt((double)n);
#pragma omp parallel for schedule(static)
  for (int64_t r = 0; r < rows; ++r) {
    double* v = x + r * n;
    if (!inverse && signs != 0)
      for (int64_t j = 0; j < n; ++j) v[j] *= (double)signs[j];
    for (int64_t h = 1; h < n; h *= 2)
      for (int64_t b = 0; b < n; b += 2 * h)
        for (int64_t j = b; j < b + h; ++j) {
          const double p = v[j], q = v[j + h];
          v[j] = p + q;
          v[j + h] = p - q;
        }
    for (int64_t j = 0; j < n; ++j) v[j] *= scale;
    if (inverse && signs != 0)
      for (int64_t j = 0; j < n; ++j) v[j] *= (double)signs[j];
  }
}

/* threads OpenMP will use for the loops above */
int oracle_threads(void) {
  int t = 1;
#pragma omp parallel
  {
#pragma omp single
    t = omp_get_num_threads();
  }
  return t;
}
