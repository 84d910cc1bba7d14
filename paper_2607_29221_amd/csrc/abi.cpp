// C ABI of libmosaic (declared in include/mosaic.h): argument validation,
// translation of mosaic_rng into kernel parameters, and dispatch to the
// kernels. Nothing here allocates device memory or keeps state between calls
// except the per-thread error message.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <string>

#include "../../include/mosaic.h"
#include "../../include/mosaic_probe.h"
#include "internal.h"

using namespace mosaic;

namespace {

thread_local std::string g_last_error;

mosaic_status fail(mosaic_status st, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
mosaic_status fail(mosaic_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

mosaic_status hip_status(hipError_t e, const char* what) {
  if (e == hipSuccess) return MOSAIC_OK;
  return fail(MOSAIC_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int64_t padded_k(int64_t k) { return 64 * ((k + 63) / 64); }

constexpr int64_t kMaxGridThreads = (int64_t(1) << 32) - 256;

// Discrete Gaussian thresholds in extended precision (see mosaic.h).
void dgauss_table(double sigma, int bound, uint64_t* out) {
  long double w[2 * kMaxDgaussBound + 1];
  long double z = 0.0L;
  for (int j = -bound; j <= bound; ++j) {
    long double p;
    if (sigma == 0.0)
      p = (j == 0) ? 1.0L : 0.0L;
    else
      p = expl(-((long double)j * (long double)j) / (2.0L * (long double)sigma * (long double)sigma));
    w[j + bound] = p;
    z += p;
  }
  long double acc = 0.0L;
  for (int k = 0; k < 2 * bound; ++k) {
    acc += w[k];
    const long double v = floorl(acc / z * 4294967296.0L + 0.5L);
    out[k] = (uint64_t)v;
  }
}

mosaic_status rng_args(const mosaic_rng* r, RngArgs* a) {
  if (r == nullptr) return fail(MOSAIC_ERR_INVALID_ARG, "rng is NULL");
  *a = RngArgs{};
  a->k0 = (uint32_t)(r->seed & 0xFFFFFFFFu);
  a->k1 = (uint32_t)(r->seed >> 32);
  a->stream = r->stream;
  a->instance = r->instance;
  a->dist = r->dist;
  a->transposed = r->transposed != 0;
  a->sparse_shift = 32;
  switch (r->dist) {
    case MOSAIC_DIST_ZERO:
    case MOSAIC_DIST_UNIFORM:
      break;
    case MOSAIC_DIST_DGAUSS:
      if (r->bound < 0 || r->bound > kMaxDgaussBound)
        return fail(MOSAIC_ERR_INVALID_ARG, "dgauss bound %d outside [0, %d]", r->bound, kMaxDgaussBound);
      if (!(r->sigma >= 0.0) || !std::isfinite(r->sigma))
        return fail(MOSAIC_ERR_INVALID_ARG, "dgauss sigma must be finite and >= 0");
      a->bound = r->bound;
      {
        uint64_t t[2 * kMaxDgaussBound];
        dgauss_table(r->sigma, r->bound, t);
        a->dg_base = -r->bound;
        a->dg_count = 0;
        for (int k = 0; k < 2 * r->bound; ++k) {
          if (t[k] == 0) ++a->dg_base;
          else if (t[k] < (1ull << 32)) a->th[a->dg_count++] = (uint32_t)t[k];
        }
      }
      break;
    case MOSAIC_DIST_SPARSE:
      if (r->log2_inv_density < 0 || r->log2_inv_density > 31)
        return fail(MOSAIC_ERR_INVALID_ARG, "sparse log2_inv_density %d outside [0, 31]", r->log2_inv_density);
      a->sparse_shift = 32 - r->log2_inv_density;
      break;
    case MOSAIC_DIST_WEIGHT:
      if (r->row_weight < 0) return fail(MOSAIC_ERR_INVALID_ARG, "row_weight %d is negative", r->row_weight);
      a->row_weight = r->row_weight;
      break;
    default:
      return fail(MOSAIC_ERR_INVALID_ARG, "unknown distribution %d", r->dist);
  }
  return MOSAIC_OK;
}

// Digit-layout operand of rows x cols; a matrix without elements may be NULL.
mosaic_status check_digits(const int8_t* p, int64_t pitch, int64_t rows, int64_t cols, const char* name) {
  if (rows == 0 || cols == 0) {
    if (pitch < 0 || pitch % 64 != 0) return fail(MOSAIC_ERR_INVALID_ARG, "%s pitch must be a multiple of 64", name);
    return MOSAIC_OK;
  }
  if (p == nullptr) return fail(MOSAIC_ERR_INVALID_ARG, "%s is NULL", name);
  if (!aligned16(p)) return fail(MOSAIC_ERR_INVALID_ARG, "%s is not 16-byte aligned", name);
  if (pitch % 64 != 0 || pitch < 4 * padded_k(cols))
    return fail(MOSAIC_ERR_INVALID_ARG, "%s pitch %lld must be a multiple of 64 and >= %lld", name,
                (long long)pitch, (long long)(4 * padded_k(cols)));
  return MOSAIC_OK;
}

// A WEIGHT stream matrix of rows x cols that the row kernels can draw.
mosaic_status check_weighted(const mosaic_rng* r, int64_t cols) {
  if (r->transposed) return fail(MOSAIC_ERR_UNSUPPORTED, "WEIGHT streams cannot be transposed");
  if (r->row_weight < 0 || r->row_weight > cols)
    return fail(MOSAIC_ERR_INVALID_ARG, "row_weight %d outside [0, cols = %lld]", r->row_weight, (long long)cols);
  if (cols > WEIGHT_MAX_COLS || r->row_weight > WEIGHT_MAX_T)
    return fail(MOSAIC_ERR_UNSUPPORTED, "WEIGHT needs cols <= %lld and row_weight <= %lld",
                (long long)WEIGHT_MAX_COLS, (long long)WEIGHT_MAX_T);
  return MOSAIC_OK;
}

// rng of the compressed-row calls: a non-transposed SPARSE or WEIGHT stream.
mosaic_status check_lpn_rng(const mosaic_rng* r, int64_t cols, RngArgs* a) {
  if (r == nullptr || (r->dist != MOSAIC_DIST_SPARSE && r->dist != MOSAIC_DIST_WEIGHT) || r->transposed)
    return fail(MOSAIC_ERR_INVALID_ARG, "rng must be a non-transposed SPARSE or WEIGHT stream");
  if (r->dist == MOSAIC_DIST_WEIGHT) {
    const mosaic_status st = check_weighted(r, cols);
    if (st != MOSAIC_OK) return st;
  }
  return rng_args(r, a);
}

}  // namespace

extern "C" {

int32_t mosaic_abi_version(void) { return MOSAIC_ABI_VERSION; }

const char* mosaic_last_error_message(void) { return g_last_error.c_str(); }

const char* mosaic_last_error_string(void) { return g_last_error.c_str(); }

mosaic_status mosaic_dgauss_thresholds(double sigma, int32_t bound, uint64_t* out) {
  if (out == nullptr) return fail(MOSAIC_ERR_INVALID_ARG, "out is NULL");
  if (bound < 0 || bound > kMaxDgaussBound)
    return fail(MOSAIC_ERR_INVALID_ARG, "bound %d outside [0, %d]", bound, kMaxDgaussBound);
  if (!(sigma >= 0.0) || !std::isfinite(sigma)) return fail(MOSAIC_ERR_INVALID_ARG, "sigma must be finite and >= 0");
  dgauss_table(sigma, bound, out);
  return MOSAIC_OK;
}

mosaic_status mosaic_mask(const void* x, int32_t x_dtype, int64_t x_rs, int64_t x_cs, const uint32_t* u,
                          int64_t ldu, const mosaic_rng* noise, int64_t rows, int64_t cols, uint32_t* out,
                          int64_t ldo, int8_t* out_dig, int64_t dig_pitch, void* stream) {
  if (rows < 0 || cols < 0) return fail(MOSAIC_ERR_INVALID_ARG, "negative size");
  if (rows == 0 || cols == 0) return MOSAIC_OK;
  if (out == nullptr && out_dig == nullptr) return fail(MOSAIC_ERR_INVALID_ARG, "no output given");
  if (x != nullptr && (x_dtype < MOSAIC_I8 || x_dtype > MOSAIC_U32))
    return fail(MOSAIC_ERR_INVALID_ARG, "unknown x_dtype %d", x_dtype);
  if (u != nullptr && ldu < cols) return fail(MOSAIC_ERR_INVALID_ARG, "ldu < cols");
  if (out != nullptr && ldo < cols) return fail(MOSAIC_ERR_INVALID_ARG, "ldo < cols");
  if (out_dig != nullptr) {
    const mosaic_status st = check_digits(out_dig, dig_pitch, rows, cols, "out_dig");
    if (st != MOSAIC_OK) return st;
  }
  MaskLaunch a{};
  a.x = x;
  a.x_dtype = x_dtype;
  a.x_rs = x_rs;
  a.x_cs = x_cs;
  a.u = u;
  a.ldu = ldu;
  a.has_noise = 0;
  if (noise != nullptr) {
    if (noise->dist == MOSAIC_DIST_WEIGHT)
      return fail(MOSAIC_ERR_UNSUPPORTED, "WEIGHT streams are drawn by mosaic_sample, not inside the mask pass");
    const mosaic_status st = rng_args(noise, &a.noise);
    if (st != MOSAIC_OK) return st;
    a.has_noise = noise->dist != MOSAIC_DIST_ZERO;
  }
  a.rows = rows;
  a.cols = cols;
  a.out = out;
  a.ldo = ldo;
  a.dig = out_dig;
  a.pitch = dig_pitch;
  const int64_t groups = out_dig ? padded_k(cols) / 16 : (cols + 15) / 16;
  if (rows > 0 && groups > kMaxGridThreads / rows) return fail(MOSAIC_ERR_UNSUPPORTED, "matrix too large for one launch");
  return hip_status(launch_mask(a, (hipStream_t)stream), "mask launch");
}

mosaic_status mosaic_sample(const mosaic_rng* rng, int64_t rows, int64_t cols, uint32_t* out, int64_t ldo,
                            int8_t* out_dig, int64_t dig_pitch, void* stream) {
  if (rng == nullptr) return fail(MOSAIC_ERR_INVALID_ARG, "rng is NULL");
  if (rng->dist != MOSAIC_DIST_WEIGHT)
    return mosaic_mask(nullptr, MOSAIC_U32, 0, 0, nullptr, 0, rng, rows, cols, out, ldo, out_dig, dig_pitch, stream);
  if (rows < 0 || cols < 0) return fail(MOSAIC_ERR_INVALID_ARG, "negative size");
  if (rows == 0 || cols == 0) return MOSAIC_OK;
  if (out == nullptr && out_dig == nullptr) return fail(MOSAIC_ERR_INVALID_ARG, "no output given");
  if (out != nullptr && ldo < cols) return fail(MOSAIC_ERR_INVALID_ARG, "ldo < cols");
  if (out_dig != nullptr) {
    const mosaic_status st = check_digits(out_dig, dig_pitch, rows, cols, "out_dig");
    if (st != MOSAIC_OK) return st;
  }
  mosaic_status st = check_weighted(rng, cols);
  if (st != MOSAIC_OK) return st;
  RngArgs a{};
  st = rng_args(rng, &a);
  if (st != MOSAIC_OK) return st;
  if (rows > 0x7FFFFFFF) return fail(MOSAIC_ERR_UNSUPPORTED, "too many rows");
  return hip_status(launch_weighted_sample(a, rows, cols, out, ldo, out_dig, dig_pitch, (hipStream_t)stream),
                    "weighted sample launch");
}

mosaic_status mosaic_sample_signs(const mosaic_rng* rng, int64_t n, int8_t* out, void* stream) {
  if (n < 0) return fail(MOSAIC_ERR_INVALID_ARG, "negative size");
  if (rng == nullptr) return fail(MOSAIC_ERR_INVALID_ARG, "rng is NULL");
  if (n == 0) return MOSAIC_OK;
  if (out == nullptr) return fail(MOSAIC_ERR_INVALID_ARG, "out is NULL");
  if (rng == nullptr) return fail(MOSAIC_ERR_INVALID_ARG, "rng is NULL");
  if (n > 4 * kMaxGridThreads) return fail(MOSAIC_ERR_UNSUPPORTED, "vector too long");
  RngArgs a{};
  a.k0 = (uint32_t)(rng->seed & 0xFFFFFFFFu);
  a.k1 = (uint32_t)(rng->seed >> 32);
  a.stream = rng->stream;
  a.instance = rng->instance;
  return hip_status(launch_signs(a, n, out, (hipStream_t)stream), "signs launch");
}

mosaic_status mosaic_masked_matmul(const int8_t* a_dig, int64_t a_pitch, const int8_t* b_dig, int64_t b_pitch,
                                   int64_t M, int64_t N, int64_t K, uint32_t* c, int64_t ldc, void* stream) {
  if (M < 0 || N < 0 || K < 0) return fail(MOSAIC_ERR_INVALID_ARG, "negative size");
  if (M == 0 || N == 0) return MOSAIC_OK;
  if (c == nullptr) return fail(MOSAIC_ERR_INVALID_ARG, "c is NULL");
  if (ldc < N) return fail(MOSAIC_ERR_INVALID_ARG, "ldc < N");
  mosaic_status st = check_digits(a_dig, a_pitch, M, K, "a_dig");
  if (st != MOSAIC_OK) return st;
  st = check_digits(b_dig, b_pitch, N, K, "b_dig");
  if (st != MOSAIC_OK) return st;
  if (a_pitch > (int64_t(1) << 23) || b_pitch > (int64_t(1) << 23))
    return fail(MOSAIC_ERR_UNSUPPORTED, "digit pitch above 8 MiB");
  GemmLaunch g{};
  g.a = a_dig;
  g.a_pitch = a_pitch;
  g.b = b_dig;
  g.b_pitch = b_pitch;
  g.M = M;
  g.N = N;
  g.c = c;
  g.ldc = ldc;
  // Inner chunks of at most MAX_K_CHUNK columns (digit columns are contiguous
  // along a row, so a chunk at column k0 starts 4 k0 bytes in): the first
  // stores, the others add.
  const int64_t Kp = padded_k(K);
  int64_t k0 = 0;
  do {
    const int64_t kc = (Kp - k0 < MAX_K_CHUNK) ? Kp - k0 : MAX_K_CHUNK;
    g.a = a_dig + 4 * k0;
    g.b = b_dig + 4 * k0;
    g.Kp = kc;
    const mosaic_status ls = hip_status(launch_ring_gemm(g, k0 == 0 ? EPI_STORE : EPI_ACCUM, (hipStream_t)stream),
                                        "ring product launch");
    if (ls != MOSAIC_OK) return ls;
    k0 += kc;
  } while (k0 < Kp);
  return MOSAIC_OK;
}

mosaic_status mosaic_masked_matmul_words(const int8_t* a_dig, int64_t a_pitch, const uint32_t* b, int64_t ldb,
                                         int64_t M, int64_t N, int64_t K, uint32_t* c, int64_t ldc,
                                         int32_t accumulate, void* stream) {
  if (M < 0 || N < 0 || K < 0) return fail(MOSAIC_ERR_INVALID_ARG, "negative size");
  if (M == 0 || N == 0) return MOSAIC_OK;
  if (c == nullptr) return fail(MOSAIC_ERR_INVALID_ARG, "c is NULL");
  if (ldc < N) return fail(MOSAIC_ERR_INVALID_ARG, "ldc < N");
  if (M > SKINNY_MAX_M) return fail(MOSAIC_ERR_UNSUPPORTED, "A must have at most %lld rows", (long long)SKINNY_MAX_M);
  mosaic_status st = check_digits(a_dig, a_pitch, M, K, "a_dig");
  if (st != MOSAIC_OK) return st;
  if (K > 0) {
    if (b == nullptr) return fail(MOSAIC_ERR_INVALID_ARG, "b is NULL");
    if (ldb < K) return fail(MOSAIC_ERR_INVALID_ARG, "ldb < K");
    if (!aligned16(b) || ldb % 4 != 0) return fail(MOSAIC_ERR_UNSUPPORTED, "b must be 16-byte aligned, ldb a multiple of 4");
  }
  if (a_pitch > (int64_t(1) << 23) || 4 * ldb > (int64_t(1) << 23))
    return fail(MOSAIC_ERR_UNSUPPORTED, "row pitch above 8 MiB");
  GemmLaunch g{};
  g.a_pitch = a_pitch;
  g.b_pitch = 4 * ldb;
  g.M = M;
  g.N = N;
  g.c = c;
  g.ldc = ldc;
  const int64_t Kp = padded_k(K);
  int64_t k0 = 0;
  do {
    const int64_t kc = (Kp - k0 < MAX_K_CHUNK) ? Kp - k0 : MAX_K_CHUNK;
    g.a = a_dig + 4 * k0;
    g.b = (const int8_t*)(b + k0);
    g.Kp = kc;
    g.b_last = 16 * ((K - k0 + 3) / 4) < 4 * kc ? 16 * ((K - k0 + 3) / 4) : 4 * kc;
    const EpilogueKind epi = (k0 == 0 && accumulate == 0) ? EPI_STORE : EPI_ACCUM;
    const mosaic_status ls = hip_status(launch_ring_gemm_words_b(g, epi, (hipStream_t)stream), "ring product launch");
    if (ls != MOSAIC_OK) return ls;
    k0 += kc;
  } while (k0 < Kp);
  return MOSAIC_OK;
}

mosaic_status mosaic_integrity_check(const int8_t* ct_dig, int64_t ct_pitch, const int8_t* a_dig, int64_t a_pitch,
                                     const int8_t* v_dig, int64_t v_pitch, const uint32_t* yq, int64_t ldyq,
                                     int64_t t, int64_t M, int64_t K, int64_t NR, uint32_t* d, int64_t ldd,
                                     int64_t* count, void* stream) {
  if (t < 0 || M < 0 || K < 0 || NR < 0) return fail(MOSAIC_ERR_INVALID_ARG, "negative size");
  if (count == nullptr) return fail(MOSAIC_ERR_INVALID_ARG, "count is NULL");
  if (t > SKINNY_MAX_M) return fail(MOSAIC_ERR_UNSUPPORTED, "at most %lld check vectors", (long long)SKINNY_MAX_M);
  const bool work = t > 0 && M > 0;
  if (work) {
    if (d == nullptr) return fail(MOSAIC_ERR_INVALID_ARG, "d is NULL");
    if (ldd < M) return fail(MOSAIC_ERR_INVALID_ARG, "ldd < M");
    mosaic_status st = check_digits(ct_dig, ct_pitch, t, K, "ct_dig");
    if (st == MOSAIC_OK) st = check_digits(a_dig, a_pitch, M, K, "a_dig");
    if (st == MOSAIC_OK) st = check_digits(v_dig, v_pitch, t, NR, "v_dig");
    if (st != MOSAIC_OK) return st;
    if (NR > 0) {
      if (yq == nullptr) return fail(MOSAIC_ERR_INVALID_ARG, "yq is NULL");
      if (ldyq < NR) return fail(MOSAIC_ERR_INVALID_ARG, "ldyq < NR");
      if (!aligned16(yq) || ldyq % 4 != 0)
        return fail(MOSAIC_ERR_UNSUPPORTED, "yq must be 16-byte aligned, ldyq a multiple of 4");
    }
    if (ct_pitch > (int64_t(1) << 23) || a_pitch > (int64_t(1) << 23) || v_pitch > (int64_t(1) << 23) ||
        4 * ldyq > (int64_t(1) << 23))
      return fail(MOSAIC_ERR_UNSUPPORTED, "row pitch above 8 MiB");
  }
  const hipStream_t s = (hipStream_t)stream;
  mosaic_status st = hip_status(launch_clear_check(d, ldd, work ? t : 0, work ? M : 0, count, s), "check clear launch");
  if (st != MOSAIC_OK || !work) return st;
  GemmLaunch g{};
  g.M = t;
  g.N = M;
  g.c = d;
  g.ldc = ldd;
  // d += c^T A'^T, in inner chunks that fit the accumulators
  g.a_pitch = ct_pitch;
  g.b_pitch = a_pitch;
  const int64_t Kp = padded_k(K);
  for (int64_t k0 = 0; k0 < Kp; k0 += MAX_K_CHUNK) {
    g.a = ct_dig + 4 * k0;
    g.b = a_dig + 4 * k0;
    g.Kp = (Kp - k0 < MAX_K_CHUNK) ? Kp - k0 : MAX_K_CHUNK;
    st = hip_status(launch_ring_gemm(g, EPI_ACCUM, s), "check product launch");
    if (st != MOSAIC_OK) return st;
  }
  // d -= V [Y' | Q]^T, B read as ring words
  g.negate = true;
  g.a_pitch = v_pitch;
  g.b_pitch = 4 * ldyq;
  const int64_t NRp = padded_k(NR);
  for (int64_t k0 = 0; k0 < NRp; k0 += MAX_K_CHUNK) {
    const int64_t kc = (NRp - k0 < MAX_K_CHUNK) ? NRp - k0 : MAX_K_CHUNK;
    g.a = v_dig + 4 * k0;
    g.b = (const int8_t*)(yq + k0);
    g.Kp = kc;
    g.b_last = 16 * ((NR - k0 + 3) / 4) < 4 * kc ? 16 * ((NR - k0 + 3) / 4) : 4 * kc;
    st = hip_status(launch_ring_gemm_words_b(g, EPI_ACCUM, s), "check product launch");
    if (st != MOSAIC_OK) return st;
  }
  return hip_status(launch_count_mismatches(d, ldd, nullptr, 0, t, M, count, s, false), "check count launch");
}

mosaic_status mosaic_rotate_quantize_mask(const float* x, int64_t ldx, int64_t rows, int64_t n, int64_t block,
                                          const int8_t* signs, int32_t qmax, const uint32_t* u, int64_t ldu,
                                          const mosaic_rng* noise, int8_t* out_dig, int64_t dig_pitch,
                                          float* scale, void* stream) {
  if (rows < 0 || n < 0) return fail(MOSAIC_ERR_INVALID_ARG, "negative size");
  if (rows == 0 || n == 0) return MOSAIC_OK;
  if (qmax < 1) return fail(MOSAIC_ERR_INVALID_ARG, "qmax must be >= 1");
  if (x == nullptr || out_dig == nullptr) return fail(MOSAIC_ERR_INVALID_ARG, "x or out_dig is NULL");
  int lg = 0;
  while (lg < 62 && (int64_t(1) << lg) < block) ++lg;
  if (block <= 0 || (int64_t(1) << lg) != block) return fail(MOSAIC_ERR_INVALID_ARG, "block must be a power of two");
  if (n % block != 0) return fail(MOSAIC_ERR_INVALID_ARG, "n must be a multiple of block");
  if (!rotate_quantize_mask_supported(lg)) return fail(MOSAIC_ERR_UNSUPPORTED, "block outside [2^10, 2^14]");
  if (scale == nullptr) return fail(MOSAIC_ERR_INVALID_ARG, "scale is NULL");
  if (ldx < n || (ldx & 3) != 0 || ((uintptr_t)x & 15) != 0)
    return fail(MOSAIC_ERR_UNSUPPORTED, "x must be 16-byte aligned with ldx >= n, a multiple of 4");
  if (u != nullptr && (ldu < n || (ldu & 3) != 0 || ((uintptr_t)u & 15) != 0))
    return fail(MOSAIC_ERR_UNSUPPORTED, "u must be 16-byte aligned with ldu >= n, a multiple of 4");
  mosaic_status st = check_digits(out_dig, dig_pitch, rows, n, "out_dig");
  if (st != MOSAIC_OK) return st;
  if (((uintptr_t)out_dig & 15) != 0) return fail(MOSAIC_ERR_UNSUPPORTED, "out_dig must be 16-byte aligned");
  RngArgs na{};
  if (noise != nullptr) {
    if (noise->transposed) return fail(MOSAIC_ERR_UNSUPPORTED, "transposed noise");
    st = rng_args(noise, &na);
    if (st != MOSAIC_OK) return st;
  }
  if (rows > 0x7FFFFFFF) return fail(MOSAIC_ERR_UNSUPPORTED, "too many rows");
  return hip_status(launch_rotate_quantize_mask(x, ldx, rows, n, lg, signs, qmax, u, ldu,
                                                noise != nullptr ? &na : nullptr, out_dig, dig_pitch, scale,
                                                (hipStream_t)stream), "rotate-quantize-mask launch");
}

mosaic_status mosaic_sparse_csr_count(const mosaic_rng* rng, int64_t rows, int64_t cols, int64_t* row_ptr,
                                      void* stream) {
  if (rows < 0 || cols < 0) return fail(MOSAIC_ERR_INVALID_ARG, "negative size");
  if (cols > 0x7FFFFFFF) return fail(MOSAIC_ERR_UNSUPPORTED, "cols must fit int32");
  if (row_ptr == nullptr) return fail(MOSAIC_ERR_INVALID_ARG, "row_ptr is NULL");
  RngArgs a{};
  mosaic_status st = check_lpn_rng(rng, cols, &a);
  if (st != MOSAIC_OK) return st;
  if (rows > 0x7FFFFFFF) return fail(MOSAIC_ERR_UNSUPPORTED, "too many rows");
  if (rng->dist == MOSAIC_DIST_WEIGHT)
    return hip_status(launch_weighted_csr_count(rows, a.row_weight, row_ptr, (hipStream_t)stream),
                      "weighted count launch");
  return hip_status(launch_sparse_csr_count(a, rows, cols, row_ptr, (hipStream_t)stream), "sparse count launch");
}

mosaic_status mosaic_sparse_csr_fill(const mosaic_rng* rng, int64_t rows, int64_t cols, const int64_t* row_ptr,
                                     int32_t* col_idx, uint32_t* values, void* stream) {
  if (rows < 0 || cols < 0) return fail(MOSAIC_ERR_INVALID_ARG, "negative size");
  if (cols > 0x7FFFFFFF) return fail(MOSAIC_ERR_UNSUPPORTED, "cols must fit int32");
  if (rows == 0 || cols == 0) return MOSAIC_OK;
  if (row_ptr == nullptr || col_idx == nullptr || values == nullptr)
    return fail(MOSAIC_ERR_INVALID_ARG, "row_ptr, col_idx or values is NULL");
  RngArgs a{};
  mosaic_status st = check_lpn_rng(rng, cols, &a);
  if (st != MOSAIC_OK) return st;
  if (rows > 0x7FFFFFFF) return fail(MOSAIC_ERR_UNSUPPORTED, "too many rows");
  if (rng->dist == MOSAIC_DIST_WEIGHT)
    return hip_status(launch_weighted_csr_fill(a, rows, cols, row_ptr, col_idx, values, (hipStream_t)stream),
                      "weighted fill launch");
  return hip_status(launch_sparse_csr_fill(a, rows, cols, row_ptr, col_idx, values, (hipStream_t)stream),
                    "sparse fill launch");
}

mosaic_status mosaic_sparse_gather_rows(int64_t rows, const int64_t* row_ptr, const int32_t* col_idx,
                                        const uint32_t* values, const uint32_t* d, int64_t ldd, int64_t ncols,
                                        uint32_t* c, int64_t ldc, int32_t subtract, void* stream) {
  if (rows < 0 || ncols < 0) return fail(MOSAIC_ERR_INVALID_ARG, "negative size");
  if (rows == 0 || ncols == 0) return MOSAIC_OK;
  if (row_ptr == nullptr || col_idx == nullptr || values == nullptr || d == nullptr || c == nullptr)
    return fail(MOSAIC_ERR_INVALID_ARG, "NULL operand");
  if (ldd < ncols || ldc < ncols) return fail(MOSAIC_ERR_INVALID_ARG, "leading dimension < ncols");
  if (rows > 0x7FFFFFFF || (ncols + 63) / 64 > 65535) return fail(MOSAIC_ERR_UNSUPPORTED, "too large for one launch");
  return hip_status(launch_sparse_gather_rows(rows, row_ptr, col_idx, values, d, ldd, ncols, c, ldc, subtract != 0,
                                              (hipStream_t)stream), "sparse gather launch");
}

mosaic_status mosaic_sparse_stream_gather_rows(const mosaic_rng* rng, int64_t rows, int64_t rcols, const uint32_t* d,
                                               int64_t ldd, int64_t ncols, uint32_t* c, int64_t ldc, int32_t subtract,
                                               void* stream) {
  if (rows < 0 || rcols < 0 || ncols < 0) return fail(MOSAIC_ERR_INVALID_ARG, "negative size");
  if (rows == 0 || ncols == 0) return MOSAIC_OK;
  if (c == nullptr || (rcols > 0 && d == nullptr)) return fail(MOSAIC_ERR_INVALID_ARG, "NULL operand");
  if (ldd < ncols || ldc < ncols) return fail(MOSAIC_ERR_INVALID_ARG, "leading dimension < ncols");
  RngArgs a{};
  mosaic_status st = check_lpn_rng(rng, rcols, &a);
  if (st != MOSAIC_OK) return st;
  if (rows > 0x7FFFFFFF || (ncols + 63) / 64 > 65535) return fail(MOSAIC_ERR_UNSUPPORTED, "too large for one launch");
  return hip_status(launch_sparse_stream_gather_rows(a, rows, rcols, d, ldd, ncols, c, ldc, subtract != 0,
                                                     (hipStream_t)stream), "sparse gather launch");
}

mosaic_status mosaic_sparse_gather_cols(int64_t M, int64_t N, const int64_t* row_ptr, const int32_t* col_idx,
                                        const uint32_t* values, const uint32_t* d, int64_t ldd, uint32_t* c,
                                        int64_t ldc, int32_t subtract, const float* s_rows, const float* s_cols,
                                        const float* bias, float* y_f32, int64_t ldf, void* stream) {
  if (M < 0 || N < 0) return fail(MOSAIC_ERR_INVALID_ARG, "negative size");
  if (M == 0 || N == 0) return MOSAIC_OK;
  if (row_ptr == nullptr || col_idx == nullptr || values == nullptr || d == nullptr || c == nullptr)
    return fail(MOSAIC_ERR_INVALID_ARG, "NULL operand");
  if (ldc < N || ldd < 0) return fail(MOSAIC_ERR_INVALID_ARG, "ldc < N");
  if (y_f32 != nullptr && (ldf < N || s_rows == nullptr || s_cols == nullptr))
    return fail(MOSAIC_ERR_INVALID_ARG, "y_f32 needs ldf >= N and both scale vectors");
  if (bias != nullptr && y_f32 == nullptr) return fail(MOSAIC_ERR_INVALID_ARG, "bias needs y_f32");
  if (M > 0x7FFFFFFF || (N + 31) / 32 > 65535) return fail(MOSAIC_ERR_UNSUPPORTED, "too large for one launch");
  const Dequant dq{s_rows, s_cols, bias, y_f32, ldf};
  return hip_status(launch_sparse_gather_cols(M, N, row_ptr, col_idx, values, d, ldd, c, ldc, subtract != 0, dq,
                                              (hipStream_t)stream), "sparse gather launch");
}

mosaic_status mosaic_count_mismatches(const uint32_t* a, int64_t lda, const uint32_t* b, int64_t ldb,
                                      int64_t rows, int64_t cols, int64_t* count, void* stream) {
  if (rows < 0 || cols < 0) return fail(MOSAIC_ERR_INVALID_ARG, "negative size");
  if (count == nullptr) return fail(MOSAIC_ERR_INVALID_ARG, "count is NULL");
  if (rows > 0 && cols > 0) {
    if (a == nullptr || b == nullptr) return fail(MOSAIC_ERR_INVALID_ARG, "a or b is NULL");
    if (lda < cols || ldb < cols) return fail(MOSAIC_ERR_INVALID_ARG, "leading dimension < cols");
  }
  return hip_status(launch_count_mismatches(a, lda, b, ldb, rows, cols, count, (hipStream_t)stream),
                    "mismatch count launch");
}

mosaic_status mosaic_unmask(const uint32_t* ym, int64_t ldy, const uint32_t* kc, int64_t ldk, const int8_t* q_dig,
                            int64_t q_pitch, const int8_t* l_dig, int64_t l_pitch, int64_t M, int64_t N, int64_t R,
                            int32_t* y, int64_t ldo, const float* s_rows, const float* s_cols, const float* bias,
                            float* y_f32, int64_t ldf, void* stream) {
  if (M < 0 || N < 0 || R < 0) return fail(MOSAIC_ERR_INVALID_ARG, "negative size");
  if (R >= 32768) return fail(MOSAIC_ERR_UNSUPPORTED, "R must be < 32768");
  if (M == 0 || N == 0) return MOSAIC_OK;
  if (ym == nullptr) return fail(MOSAIC_ERR_INVALID_ARG, "ym is NULL");
  if (ldy < N) return fail(MOSAIC_ERR_INVALID_ARG, "ldy < N");
  if (kc != nullptr && ldk < N) return fail(MOSAIC_ERR_INVALID_ARG, "ldk < N");
  if (y == nullptr && y_f32 == nullptr) return fail(MOSAIC_ERR_INVALID_ARG, "no output given");
  if (y != nullptr && ldo < N) return fail(MOSAIC_ERR_INVALID_ARG, "ldo < N");
  if (y_f32 != nullptr && (ldf < N || s_rows == nullptr || s_cols == nullptr))
    return fail(MOSAIC_ERR_INVALID_ARG, "y_f32 needs ldf >= N and both scale vectors");
  if (bias != nullptr && y_f32 == nullptr) return fail(MOSAIC_ERR_INVALID_ARG, "bias needs y_f32");
  GemmLaunch g{};
  g.M = M;
  g.N = N;
  g.ym = ym;
  g.ldy = ldy;
  g.kc = kc;
  g.ldk = ldk;
  g.y = y;
  g.ldo = ldo;
  g.s_rows = s_rows;
  g.s_cols = s_cols;
  g.bias = bias;
  g.y_f32 = y_f32;
  g.ldf = ldf;
  if (R == 0) {
    if (M > 0 && N > kMaxGridThreads / M) return fail(MOSAIC_ERR_UNSUPPORTED, "matrix too large for one launch");
    return hip_status(launch_unmask_elementwise(g, (hipStream_t)stream), "unmask launch");
  }
  mosaic_status st = check_digits(q_dig, q_pitch, M, R, "q_dig");
  if (st != MOSAIC_OK) return st;
  st = check_digits(l_dig, l_pitch, N, R, "l_dig");
  if (st != MOSAIC_OK) return st;
  if (q_pitch > (int64_t(1) << 23) || l_pitch > (int64_t(1) << 23))
    return fail(MOSAIC_ERR_UNSUPPORTED, "digit pitch above 8 MiB");
  g.a = q_dig;
  g.a_pitch = q_pitch;
  g.b = l_dig;
  g.b_pitch = l_pitch;
  g.Kp = padded_k(R);
  return hip_status(launch_ring_gemm(g, EPI_UNMASK, (hipStream_t)stream), "unmask launch");
}

mosaic_status mosaic_unmask_words(const uint32_t* ym, int64_t ldy, const uint32_t* kc, int64_t ldk, const uint32_t* q,
                                  int64_t ldq, const int8_t* l_dig, int64_t l_pitch, int64_t M, int64_t N, int64_t R,
                                  int32_t* y, int64_t ldo, const float* s_rows, const float* s_cols,
                                  const float* bias, float* y_f32, int64_t ldf, void* stream) {
  if (M < 0 || N < 0 || R < 0) return fail(MOSAIC_ERR_INVALID_ARG, "negative size");
  if (M > 16) return fail(MOSAIC_ERR_UNSUPPORTED, "q as ring words needs M <= 16");
  if (R >= 32768) return fail(MOSAIC_ERR_UNSUPPORTED, "R must be < 32768");
  if (M == 0 || N == 0) return MOSAIC_OK;
  if (ym == nullptr) return fail(MOSAIC_ERR_INVALID_ARG, "ym is NULL");
  if (ldy < N) return fail(MOSAIC_ERR_INVALID_ARG, "ldy < N");
  if (kc != nullptr && ldk < N) return fail(MOSAIC_ERR_INVALID_ARG, "ldk < N");
  if (y == nullptr && y_f32 == nullptr) return fail(MOSAIC_ERR_INVALID_ARG, "no output given");
  if (y != nullptr && ldo < N) return fail(MOSAIC_ERR_INVALID_ARG, "ldo < N");
  if (y_f32 != nullptr && (ldf < N || s_rows == nullptr || s_cols == nullptr))
    return fail(MOSAIC_ERR_INVALID_ARG, "y_f32 needs ldf >= N and both scale vectors");
  if (bias != nullptr && y_f32 == nullptr) return fail(MOSAIC_ERR_INVALID_ARG, "bias needs y_f32");
  GemmLaunch g{};
  g.M = M;
  g.N = N;
  g.ym = ym;
  g.ldy = ldy;
  g.kc = kc;
  g.ldk = ldk;
  g.y = y;
  g.ldo = ldo;
  g.s_rows = s_rows;
  g.s_cols = s_cols;
  g.bias = bias;
  g.y_f32 = y_f32;
  g.ldf = ldf;
  if (R > 0) {
    if (q == nullptr) return fail(MOSAIC_ERR_INVALID_ARG, "q is NULL");
    if (ldq < R) return fail(MOSAIC_ERR_INVALID_ARG, "ldq < R");
    if (!aligned16(q) || ldq % 4 != 0) return fail(MOSAIC_ERR_UNSUPPORTED, "q must be 16-byte aligned, ldq a multiple of 4");
    if (ldq > (int64_t(1) << 21)) return fail(MOSAIC_ERR_UNSUPPORTED, "q pitch above 8 MiB");
    const mosaic_status st = check_digits(l_dig, l_pitch, N, R, "l_dig");
    if (st != MOSAIC_OK) return st;
    if (l_pitch > (int64_t(1) << 23)) return fail(MOSAIC_ERR_UNSUPPORTED, "digit pitch above 8 MiB");
    g.a = (const int8_t*)q;
    g.a_pitch = 4 * ldq;
    g.a_last = 16 * ((R + 3) / 4);   // q's last row up to its 16-byte chunk
    g.b = l_dig;
    g.b_pitch = l_pitch;
    g.Kp = padded_k(R);
  } else if (M > 0 && N > kMaxGridThreads / M) {
    return fail(MOSAIC_ERR_UNSUPPORTED, "matrix too large for one launch");
  }
  return hip_status(launch_unmask_words_a(g, (hipStream_t)stream), "unmask launch");
}

mosaic_status mosaic_hadamard_rotate(const float* x, int64_t ldx, float* y, int64_t ldy, int64_t rows, int64_t n,
                                     int64_t block, const int8_t* signs, int32_t inverse, void* stream) {
  if (rows < 0 || n < 0) return fail(MOSAIC_ERR_INVALID_ARG, "negative size");
  if (rows == 0 || n == 0) return MOSAIC_OK;
  if (x == nullptr || y == nullptr) return fail(MOSAIC_ERR_INVALID_ARG, "x or y is NULL");
  if (!aligned16(x) || !aligned16(y)) return fail(MOSAIC_ERR_INVALID_ARG, "x and y must be 16-byte aligned");
  if (block < 16 || block > 32768 || (block & (block - 1)) != 0)
    return fail(MOSAIC_ERR_UNSUPPORTED, "block %lld must be a power of two in [16, 32768]", (long long)block);
  if (n % block != 0) return fail(MOSAIC_ERR_INVALID_ARG, "n must be a multiple of block");
  if (ldx < n || ldy < n || ldx % 4 != 0 || ldy % 4 != 0)
    return fail(MOSAIC_ERR_INVALID_ARG, "ldx and ldy must be >= n and multiples of 4");
  if (signs != nullptr && !aligned16(signs)) return fail(MOSAIC_ERR_INVALID_ARG, "signs must be 16-byte aligned");
  if (rows > 0 && n > 0) {
    const char* xb = (const char*)x;
    const char* xe = (const char*)(x + (rows - 1) * ldx + n);
    const char* yb = (const char*)y;
    const char* ye = (const char*)(y + (rows - 1) * ldy + n);
    if ((const float*)x != y && xb < ye && yb < xe) return fail(MOSAIC_ERR_INVALID_ARG, "x and y overlap");
    if ((const float*)x == y && ldx != ldy) return fail(MOSAIC_ERR_INVALID_ARG, "in place needs ldx == ldy");
  }
  const int64_t blocks = rows * (n / (block > 0 ? block : 1));
  if (blocks >= (int64_t(1) << 31)) return fail(MOSAIC_ERR_UNSUPPORTED, "too many blocks");
  int lb = 0;
  while ((int64_t(1) << lb) < block) ++lb;
  return hip_status(launch_hadamard(x, ldx, y, ldy, rows, n, lb, signs, inverse != 0, (hipStream_t)stream),
                    "hadamard launch");
}

mosaic_status mosaic_hadamard28_rotate(const float* x, int64_t ldx, float* y, int64_t ldy, int64_t rows, int64_t n,
                                       const int8_t* signs, int32_t inverse, void* stream) {
  if (rows < 0 || n < 0) return fail(MOSAIC_ERR_INVALID_ARG, "negative size");
  if (rows == 0 || n == 0) return MOSAIC_OK;
  if (x == nullptr || y == nullptr) return fail(MOSAIC_ERR_INVALID_ARG, "x or y is NULL");
  if (!aligned16(x) || !aligned16(y)) return fail(MOSAIC_ERR_INVALID_ARG, "x and y must be 16-byte aligned");
  const int64_t b = n / 28;
  int lb = 0;
  while ((int64_t(1) << lb) < b) ++lb;
  if (n % 28 != 0 || (int64_t(1) << lb) != b || !hadamard28_supported(lb))
    return fail(MOSAIC_ERR_UNSUPPORTED, "n = %lld must be 28 b with b in {256, 512, 1024}", (long long)n);
  if (ldx < n || ldy < n || ldx % 4 != 0 || ldy % 4 != 0)
    return fail(MOSAIC_ERR_INVALID_ARG, "ldx and ldy must be >= n and multiples of 4");
  if (signs != nullptr && !aligned16(signs)) return fail(MOSAIC_ERR_INVALID_ARG, "signs must be 16-byte aligned");
  if (rows >= (int64_t(1) << 31)) return fail(MOSAIC_ERR_UNSUPPORTED, "too many rows");
  {
    const char* xb = (const char*)x;
    const char* xe = (const char*)(x + (rows - 1) * ldx + n);
    const char* yb = (const char*)y;
    const char* ye = (const char*)(y + (rows - 1) * ldy + n);
    if ((const float*)x != y && xb < ye && yb < xe) return fail(MOSAIC_ERR_INVALID_ARG, "x and y overlap");
    if ((const float*)x == y && ldx != ldy) return fail(MOSAIC_ERR_INVALID_ARG, "in place needs ldx == ldy");
  }
  return hip_status(launch_hadamard28(x, ldx, y, ldy, rows, lb, signs, inverse != 0, (hipStream_t)stream),
                    "hadamard28 launch");
}

mosaic_status mosaic_quantize_rows(const float* x, int64_t ldx, int64_t rows, int64_t n, int32_t qmax, int32_t* q,
                                   int64_t ldq, int8_t* q_dig, int64_t q_pitch, float* scale, void* stream) {
  if (rows < 0 || n < 0) return fail(MOSAIC_ERR_INVALID_ARG, "negative size");
  if (rows == 0 || n == 0) return MOSAIC_OK;
  if (x == nullptr) return fail(MOSAIC_ERR_INVALID_ARG, "x is NULL");
  if (ldx < n) return fail(MOSAIC_ERR_INVALID_ARG, "ldx < n");
  if (qmax < 1 || qmax > (1 << 24)) return fail(MOSAIC_ERR_INVALID_ARG, "qmax outside [1, 2^24]");
  if (q == nullptr && q_dig == nullptr) return fail(MOSAIC_ERR_INVALID_ARG, "no output given");
  if (q != nullptr && ldq < n) return fail(MOSAIC_ERR_INVALID_ARG, "ldq < n");
  if (q_dig != nullptr) {
    const mosaic_status st = check_digits(q_dig, q_pitch, rows, n, "q_dig");
    if (st != MOSAIC_OK) return st;
  }
  if (rows >= (int64_t(1) << 31)) return fail(MOSAIC_ERR_UNSUPPORTED, "too many rows");
  return hip_status(launch_quantize_rows(x, ldx, rows, n, qmax, q, ldq, q_dig, q_pitch, scale, (hipStream_t)stream),
                    "quantize launch");
}

mosaic_status mosaic_probe_mfma_i8(int32_t mode, int64_t iters, int32_t* out, int64_t* ops, void* stream) {
  if (mode < 0 || mode > 2) return fail(MOSAIC_ERR_INVALID_ARG, "mode %d outside {0, 1, 2}", mode);
  if (iters < 1) return fail(MOSAIC_ERR_INVALID_ARG, "iters must be >= 1");
  if (out == nullptr || ops == nullptr) return fail(MOSAIC_ERR_INVALID_ARG, "out or ops is NULL");
  return hip_status(launch_mfma_probe(mode, iters, out, ops, (hipStream_t)stream), "mfma probe launch");
}

}  // extern "C"
