/* Driver of the oracle's C leg under AddressSanitizer and
 * UndefinedBehaviorSanitizer (tests/test_abi_sanitize.py): stream words
 * across OpenMP slices and a counter past 2^32 blocks (one call must equal
 * two calls that split the range), a small ring product against its
 * definition, and a round trip of the rotation. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

void oracle_stream_words(uint64_t seed, uint32_t stream, uint32_t instance, uint64_t t0, uint64_t count,
                         uint32_t* out);
void oracle_ring_matmul_nt(const uint32_t* A, int64_t lda, const uint32_t* B, int64_t ldb, uint32_t* C,
                           int64_t ldc, int64_t m, int64_t n, int64_t k);
void oracle_rotate_rows(double* x, int64_t rows, int64_t n, const int8_t* signs, int inverse);
int oracle_threads(void);

int main(void) {
  int fail = 0;
  const uint64_t n = 200003, t0 = 4ull * 4294967296ull - 6;
  uint32_t* a = malloc(n * 4);
  uint32_t* b = malloc(n * 4);
  oracle_stream_words(0xFFFFFFFFFFFFFFFFull, 3, 7, t0, n, a);
  oracle_stream_words(0xFFFFFFFFFFFFFFFFull, 3, 7, t0, 70001, b);
  oracle_stream_words(0xFFFFFFFFFFFFFFFFull, 3, 7, t0 + 70001, n - 70001, b + 70001);
  for (uint64_t i = 0; i < n; ++i) fail += a[i] != b[i];
  uint32_t A[3 * 5], B[4 * 5], C[3 * 4];
  for (int i = 0; i < 15; ++i) A[i] = a[i];
  for (int i = 0; i < 20; ++i) B[i] = a[100 + i];
  oracle_ring_matmul_nt(A, 5, B, 5, C, 4, 3, 4, 5);
  for (int i = 0; i < 3; ++i)
    for (int j = 0; j < 4; ++j) {
      uint64_t s = 0;
      for (int t = 0; t < 5; ++t) s += (uint64_t)A[i * 5 + t] * B[j * 5 + t];
      fail += C[i * 4 + j] != (uint32_t)s;
    }
  double x[4 * 256], y[4 * 256];
  int8_t sg[256];
  for (int i = 0; i < 1024; ++i) x[i] = y[i] = (double)(a[i] % 1000) - 500.0;
  for (int j = 0; j < 256; ++j) sg[j] = (a[2000 + j] >> 31) ? -1 : 1;
  oracle_rotate_rows(y, 4, 256, sg, 0);
  oracle_rotate_rows(y, 4, 256, sg, 1);
  for (int i = 0; i < 1024; ++i) fail += fabs(y[i] - x[i]) > 1e-9;
  fail += oracle_threads() < 1;
  free(a);
  free(b);
  printf("%s (%d failures)\n", fail ? "FAIL" : "PASS", fail);
  return fail ? 1 : 0;
}
