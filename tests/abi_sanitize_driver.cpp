// Driver of the sanitizer build (tests/test_abi_sanitize.py): calls every
// entry point of include/mosaic.h with arguments that validation must reject
// (fake device addresses that are never dereferenced), zero-sized calls that
// must do nothing, and the host-only threshold computation, under
// AddressSanitizer and UndefinedBehaviorSanitizer. Launchers are stubs that
// count calls: none may be reached.
#include <cstdint>
#include <cstdio>
#include <cstdlib>

#include "../include/mosaic.h"
#include "../include/mosaic_probe.h"

extern int g_launches;

static int g_fail = 0;
#define EXPECT(call, want)                                                                   \
  do {                                                                                       \
    const int got_ = (int)(call);                                                            \
    if (got_ != (int)(want)) {                                                               \
      std::printf("line %d: %s returned %d, expected %d (%s)\n", __LINE__, #call, got_,     \
                  (int)(want), mosaic_last_error_message());                                 \
      ++g_fail;                                                                              \
    }                                                                                        \
  } while (0)

int main() {
  const int INV = MOSAIC_ERR_INVALID_ARG, UNS = MOSAIC_ERR_UNSUPPORTED, OK = MOSAIC_OK;
  void* F = (void*)(uintptr_t)(1u << 20);
  uint32_t* Fu = (uint32_t*)F;
  int8_t* Fd = (int8_t*)F;
  float* Ff = (float*)F;
  mosaic_rng u{};
  u.seed = 1; u.stream = 2; u.instance = 3; u.dist = MOSAIC_DIST_UNIFORM;
  mosaic_rng w = u;
  w.dist = MOSAIC_DIST_WEIGHT; w.row_weight = 5;

  EXPECT(mosaic_abi_version(), MOSAIC_ABI_VERSION);
  uint64_t th[32];
  for (int b = 0; b <= 15; ++b) EXPECT(mosaic_dgauss_thresholds(0.5 + b, b, th), OK);
  EXPECT(mosaic_dgauss_thresholds(0.5, 16, th), INV);
  EXPECT(mosaic_dgauss_thresholds(-1.0, 4, th), INV);

  // sample / mask
  EXPECT(mosaic_sample(nullptr, 4, 4, Fu, 4, nullptr, 0, nullptr), INV);
  EXPECT(mosaic_sample(&u, 4, 4, nullptr, 0, nullptr, 0, nullptr), INV);
  EXPECT(mosaic_sample(&u, 4, 4, Fu, 3, nullptr, 0, nullptr), INV);
  EXPECT(mosaic_sample(&u, 4, 4, nullptr, 0, Fd, 100, nullptr), INV);
  EXPECT(mosaic_sample(&w, 4, 4, Fu, 4, nullptr, 0, nullptr), INV);               // t > cols
  mosaic_rng wt = w; wt.transposed = 1;
  EXPECT(mosaic_sample(&wt, 4, 8, Fu, 8, nullptr, 0, nullptr), UNS);
  EXPECT(mosaic_sample(&w, 4, 10000, Fu, 10000, nullptr, 0, nullptr), UNS);        // cols > 8192
  mosaic_rng bad = u; bad.dist = 9;
  EXPECT(mosaic_sample(&bad, 4, 4, Fu, 4, nullptr, 0, nullptr), INV);
  mosaic_rng dg = u; dg.dist = MOSAIC_DIST_DGAUSS; dg.bound = 16;
  EXPECT(mosaic_sample(&dg, 4, 4, Fu, 4, nullptr, 0, nullptr), INV);
  mosaic_rng sp = u; sp.dist = MOSAIC_DIST_SPARSE; sp.log2_inv_density = 32;
  EXPECT(mosaic_sample(&sp, 4, 4, Fu, 4, nullptr, 0, nullptr), INV);
  EXPECT(mosaic_mask(F, 7, 4, 1, nullptr, 0, nullptr, 4, 4, Fu, 4, nullptr, 0, nullptr), INV);
  EXPECT(mosaic_mask(F, MOSAIC_I8, 4, 1, Fu, 3, nullptr, 4, 4, Fu, 4, nullptr, 0, nullptr), INV);
  EXPECT(mosaic_mask(F, MOSAIC_I8, 4, 1, nullptr, 0, &w, 4, 8, Fu, 8, nullptr, 0, nullptr), UNS);
  EXPECT(mosaic_mask(F, MOSAIC_I8, 4, 1, nullptr, 0, nullptr, -1, 4, Fu, 4, nullptr, 0, nullptr), INV);
  EXPECT(mosaic_mask(F, MOSAIC_I8, 4, 1, nullptr, 0, nullptr, 0, 4, Fu, 4, nullptr, 0, nullptr), OK);
  EXPECT(mosaic_sample_signs(&u, 4, nullptr, nullptr), INV);
  EXPECT(mosaic_sample_signs(&u, -1, Fd, nullptr), INV);

  // products
  EXPECT(mosaic_masked_matmul(Fd, 256, Fd, 256, 4, 4, 64, nullptr, 4, nullptr), INV);
  EXPECT(mosaic_masked_matmul(Fd, 256, Fd, 256, 4, 4, 64, Fu, 3, nullptr), INV);
  EXPECT(mosaic_masked_matmul(Fd, 100, Fd, 256, 4, 4, 64, Fu, 4, nullptr), INV);
  EXPECT(mosaic_masked_matmul(Fd, 192, Fd, 256, 4, 4, 64, Fu, 4, nullptr), INV);
  EXPECT(mosaic_masked_matmul(Fd + 1, 256, Fd, 256, 4, 4, 64, Fu, 4, nullptr), INV);
  EXPECT(mosaic_masked_matmul(Fd, int64_t(1) << 24, Fd, 256, 4, 4, 64, Fu, 4, nullptr), UNS);
  EXPECT(mosaic_masked_matmul(Fd, 256, Fd, 256, -1, 4, 64, Fu, 4, nullptr), INV);
  EXPECT(mosaic_masked_matmul(Fd, 256, Fd, 256, 0, 4, 64, Fu, 4, nullptr), OK);
  EXPECT(mosaic_masked_matmul_words(Fd, 256, Fu, 64, 65, 4, 64, Fu, 4, 0, nullptr), UNS);     // M > 64
  EXPECT(mosaic_masked_matmul_words(Fd, 256, Fu, 63, 4, 4, 64, Fu, 4, 0, nullptr), INV);      // ldb < K
  EXPECT(mosaic_masked_matmul_words(Fd, 256, Fu, 66, 4, 4, 64, Fu, 4, 0, nullptr), UNS);      // ldb % 4
  EXPECT(mosaic_masked_matmul_words(Fd, 256, Fu + 1, 64, 4, 4, 64, Fu, 4, 0, nullptr), UNS);  // alignment
  EXPECT(mosaic_masked_matmul_words(Fd, 256, nullptr, 64, 4, 4, 64, Fu, 4, 0, nullptr), INV);
  EXPECT(mosaic_masked_matmul_words(Fd, 256, Fu, 64, 4, 4, 64, nullptr, 4, 0, nullptr), INV);
  int64_t* Fc = (int64_t*)F;
  EXPECT(mosaic_integrity_check(Fd, 256, Fd, 256, Fd, 256, Fu, 64, 4, 4, 64, 64, Fu, 4, nullptr, nullptr), INV);
  EXPECT(mosaic_integrity_check(Fd, 256, Fd, 256, Fd, 256, Fu, 64, 65, 4, 64, 64, Fu, 4, Fc, nullptr), UNS);
  EXPECT(mosaic_integrity_check(Fd, 256, Fd, 256, Fd, 256, Fu, 64, 4, -1, 64, 64, Fu, 4, Fc, nullptr), INV);
  EXPECT(mosaic_integrity_check(Fd, 256, Fd, 256, Fd, 256, Fu, 64, 4, 4, 64, 64, nullptr, 4, Fc, nullptr), INV);
  EXPECT(mosaic_integrity_check(Fd, 256, Fd, 256, Fd, 256, Fu, 64, 4, 4, 64, 64, Fu, 3, Fc, nullptr), INV);
  EXPECT(mosaic_integrity_check(Fd + 1, 256, Fd, 256, Fd, 256, Fu, 64, 4, 4, 64, 64, Fu, 4, Fc, nullptr), INV);
  EXPECT(mosaic_integrity_check(Fd, 256, Fd, 192, Fd, 256, Fu, 64, 4, 4, 64, 64, Fu, 4, Fc, nullptr), INV);
  EXPECT(mosaic_integrity_check(Fd, 256, Fd, 256, Fd, 256, nullptr, 64, 4, 4, 64, 64, Fu, 4, Fc, nullptr), INV);
  EXPECT(mosaic_integrity_check(Fd, 256, Fd, 256, Fd, 256, Fu, 60, 4, 4, 64, 64, Fu, 4, Fc, nullptr), INV);
  EXPECT(mosaic_integrity_check(Fd, 256, Fd, 256, Fd, 256, Fu + 1, 64, 4, 4, 64, 64, Fu, 4, Fc, nullptr), UNS);
  EXPECT(mosaic_integrity_check(Fd, 256, Fd, 256, Fd, 256, Fu, 66, 4, 4, 64, 64, Fu, 4, Fc, nullptr), UNS);
  EXPECT(mosaic_integrity_check(Fd, 256, Fd, int64_t(1) << 24, Fd, 256, Fu, 64, 4, 4, 64, 64, Fu, 4, Fc, nullptr),
         UNS);
  EXPECT(mosaic_unmask(Fu, 4, nullptr, 0, Fd, 256, Fd, 256, 4, 4, 32768, (int32_t*)F, 4, nullptr, nullptr,
                       nullptr, nullptr, 0, nullptr), UNS);
  EXPECT(mosaic_unmask(nullptr, 4, nullptr, 0, Fd, 256, Fd, 256, 4, 4, 64, (int32_t*)F, 4, nullptr, nullptr,
                       nullptr, nullptr, 0, nullptr), INV);
  EXPECT(mosaic_unmask(Fu, 4, nullptr, 0, Fd, 256, Fd, 256, 4, 4, 64, nullptr, 4, nullptr, nullptr, nullptr,
                       nullptr, 0, nullptr), INV);
  EXPECT(mosaic_unmask(Fu, 4, nullptr, 0, Fd, 256, Fd, 256, 4, 4, 64, nullptr, 4, nullptr, nullptr, nullptr, Ff,
                       4, nullptr), INV);
  EXPECT(mosaic_unmask(Fu, 4, Fu, 3, Fd, 256, Fd, 256, 4, 4, 64, (int32_t*)F, 4, nullptr, nullptr, nullptr,
                       nullptr, 0, nullptr), INV);
  EXPECT(mosaic_unmask(Fu, 4, nullptr, 0, Fd, 256, Fd, 256, 4, 4, 64, (int32_t*)F, 4, nullptr, nullptr, Ff,
                       nullptr, 0, nullptr), INV);     // bias without y_f32
  EXPECT(mosaic_unmask_words(Fu, 4, nullptr, 0, Fu, 64, Fd, 256, 17, 4, 64, (int32_t*)F, 4, nullptr, nullptr,
                             nullptr, nullptr, 0, nullptr), UNS);     // more than 16 rows
  EXPECT(mosaic_unmask_words(Fu, 4, nullptr, 0, Fu, 64, Fd, 256, 4, 4, 32768, (int32_t*)F, 4, nullptr, nullptr,
                             nullptr, nullptr, 0, nullptr), UNS);
  EXPECT(mosaic_unmask_words(Fu, 4, nullptr, 0, nullptr, 64, Fd, 256, 4, 4, 64, (int32_t*)F, 4, nullptr, nullptr,
                             nullptr, nullptr, 0, nullptr), INV);     // q missing
  EXPECT(mosaic_unmask_words(Fu, 4, nullptr, 0, Fu, 60, Fd, 256, 4, 4, 64, (int32_t*)F, 4, nullptr, nullptr,
                             nullptr, nullptr, 0, nullptr), INV);     // ldq < R
  EXPECT(mosaic_unmask_words(Fu, 4, nullptr, 0, Fu + 1, 64, Fd, 256, 4, 4, 64, (int32_t*)F, 4, nullptr, nullptr,
                             nullptr, nullptr, 0, nullptr), UNS);     // q not 16-byte aligned
  EXPECT(mosaic_unmask_words(Fu, 4, nullptr, 0, Fu, 66, Fd, 256, 4, 4, 64, (int32_t*)F, 4, nullptr, nullptr,
                             nullptr, nullptr, 0, nullptr), UNS);     // ldq not a multiple of 4
  EXPECT(mosaic_unmask_words(Fu, 4, nullptr, 0, Fu, 64, Fd, 192, 4, 4, 64, (int32_t*)F, 4, nullptr, nullptr,
                             nullptr, nullptr, 0, nullptr), INV);     // l pitch below its padded row
  EXPECT(mosaic_unmask_words(Fu, 4, nullptr, 0, Fu, 64, Fd, 256, 4, 4, 64, nullptr, 4, nullptr, nullptr, nullptr,
                             nullptr, 0, nullptr), INV);              // no output
  EXPECT(mosaic_unmask_words(Fu, 4, nullptr, 0, Fu, 64, Fd, 256, 4, 4, 64, (int32_t*)F, 4, nullptr, nullptr, Ff,
                             nullptr, 0, nullptr), INV);     // bias without y_f32

  // rotation and quantisation
  EXPECT(mosaic_hadamard_rotate(Ff, 64, Ff, 64, 4, 64, 48, nullptr, 0, nullptr), UNS);
  EXPECT(mosaic_hadamard_rotate(Ff, 64, Ff, 64, 4, 96, 64, nullptr, 0, nullptr), INV);
  EXPECT(mosaic_hadamard_rotate(Ff + 1, 64, Ff, 64, 4, 64, 64, nullptr, 0, nullptr), INV);
  EXPECT(mosaic_hadamard_rotate(Ff, 64, Ff + 4, 64, 4, 64, 64, nullptr, 0, nullptr), INV);     // overlap
  EXPECT(mosaic_hadamard_rotate(Ff, 64, Ff, 68, 4, 64, 64, nullptr, 0, nullptr), INV);         // in place, ld differ
  EXPECT(mosaic_hadamard28_rotate(Ff, 28672, Ff, 28672, 4, 28000, nullptr, 0, nullptr), UNS);
  EXPECT(mosaic_quantize_rows(Ff, 64, 4, 64, 0, (int32_t*)F, 64, nullptr, 0, nullptr, nullptr), INV);
  EXPECT(mosaic_quantize_rows(Ff, 64, 4, 64, 127, nullptr, 0, nullptr, 0, nullptr, nullptr), INV);
  EXPECT(mosaic_rotate_quantize_mask(Ff, 1024, 2, 1024, 512, nullptr, 127, nullptr, 0, nullptr, Fd, 4096, Ff,
                                     nullptr), UNS);
  EXPECT(mosaic_rotate_quantize_mask(Ff, 1024, 2, 1024, 1024, nullptr, 127, nullptr, 0, nullptr, Fd, 4096,
                                     nullptr, nullptr), INV);

  // sparse LPN and the check
  int64_t* Fl = (int64_t*)F;
  EXPECT(mosaic_sparse_csr_count(&u, 4, 4, Fl, nullptr), INV);                      // not SPARSE/WEIGHT
  EXPECT(mosaic_sparse_csr_count(&w, 4, 4, Fl, nullptr), INV);                      // t > cols
  EXPECT(mosaic_sparse_csr_fill(&sp, 4, 4, Fl, nullptr, Fu, nullptr), INV);
  EXPECT(mosaic_sparse_gather_rows(4, Fl, (int32_t*)F, Fu, Fu, 3, 4, Fu, 4, 0, nullptr), INV);
  EXPECT(mosaic_sparse_stream_gather_rows(&u, 4, 8, Fu, 4, 4, Fu, 4, 0, nullptr), INV);
  EXPECT(mosaic_sparse_gather_cols(4, 4, Fl, (int32_t*)F, Fu, Fu, 4, Fu, 3, 0, nullptr, nullptr, nullptr, nullptr, 0,
                                   nullptr), INV);
  EXPECT(mosaic_sparse_gather_cols(4, 4, Fl, (int32_t*)F, Fu, Fu, 4, Fu, 4, 0, nullptr, Ff, nullptr, Ff, 4,
                                   nullptr), INV);     // y_f32 without s_rows
  EXPECT(mosaic_sparse_gather_cols(4, 4, Fl, (int32_t*)F, Fu, Fu, 4, Fu, 4, 0, Ff, Ff, nullptr, Ff, 3,
                                   nullptr), INV);     // ldf < N
  EXPECT(mosaic_sparse_gather_cols(4, 4, Fl, (int32_t*)F, Fu, Fu, 4, Fu, 4, 0, nullptr, nullptr, Ff, nullptr, 0,
                                   nullptr), INV);     // bias without y_f32
  EXPECT(mosaic_count_mismatches(Fu, 4, Fu, 4, 4, 4, nullptr, nullptr), INV);
  EXPECT(mosaic_count_mismatches(Fu, 3, Fu, 4, 4, 4, Fl, nullptr), INV);
  int64_t ops = 0;
  EXPECT(mosaic_probe_mfma_i8(3, 10, (int32_t*)F, &ops, nullptr), INV);
  EXPECT(mosaic_probe_mfma_i8(0, 0, (int32_t*)F, &ops, nullptr), INV);

  if (g_launches != 0) {
    std::printf("%d launcher(s) reached\n", g_launches);
    ++g_fail;
  }
  std::printf("%s (%d failures)\n", g_fail ? "FAIL" : "PASS", g_fail);
  return g_fail ? 1 : 0;
}
