// Launch interfaces between the C ABI layer (abi.cpp) and the kernel files.
// Every launcher assumes its arguments were validated by the ABI layer.
#pragma once

#include <atomic>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "device_common.h"

namespace mosaic {

struct MaskLaunch {
  const void* x;
  int32_t x_dtype;        // mosaic_dtype
  int64_t x_rs, x_cs;
  const uint32_t* u;
  int64_t ldu;
  int32_t has_noise;
  RngArgs noise;
  int64_t rows, cols;
  uint32_t* out;
  int64_t ldo;
  int8_t* dig;
  int64_t pitch;
};
hipError_t launch_mask(const MaskLaunch& a, hipStream_t s);

hipError_t launch_signs(const RngArgs& r, int64_t n, int8_t* out, hipStream_t s);

hipError_t launch_sparse_csr_count(const RngArgs& r, int64_t rows, int64_t cols, int64_t* row_ptr, hipStream_t s);
hipError_t launch_sparse_csr_fill(const RngArgs& r, int64_t rows, int64_t cols, const int64_t* row_ptr,
                                  int32_t* col_idx, uint32_t* values, hipStream_t s);
hipError_t launch_sparse_gather_rows(int64_t rows, const int64_t* row_ptr, const int32_t* col_idx,
                                     const uint32_t* values, const uint32_t* d, int64_t ldd, int64_t ncols,
                                     uint32_t* c, int64_t ldc, int subtract, hipStream_t s);
hipError_t launch_sparse_stream_gather_rows(const RngArgs& r, int64_t rows, int64_t rcols, const uint32_t* d,
                                            int64_t ldd, int64_t ncols, uint32_t* c, int64_t ldc, int subtract,
                                            hipStream_t s);
// Dequantised copy of a finished ring result: y[m, n] = (float)(int32)c *
// s_rows[m] * s_cols[n] (+ bias[n]); y null for none.
struct Dequant {
  const float* s_rows;
  const float* s_cols;
  const float* bias;
  float* y;
  int64_t ld;
};
hipError_t launch_sparse_gather_cols(int64_t M, int64_t N, const int64_t* row_ptr, const int32_t* col_idx,
                                     const uint32_t* values, const uint32_t* d, int64_t ldd, uint32_t* c,
                                     int64_t ldc, int subtract, const Dequant& dq, hipStream_t s);

// Fixed-row-weight (WEIGHT) streams: at most WEIGHT_MAX_COLS columns (the
// row's permutation lives in LDS) and, where a row is staged whole in LDS,
// WEIGHT_MAX_T entries.
constexpr int64_t WEIGHT_MAX_COLS = 8192;
constexpr int64_t WEIGHT_MAX_T = 2048;
hipError_t launch_weighted_sample(const RngArgs& r, int64_t rows, int64_t cols, uint32_t* out, int64_t ldo,
                                  int8_t* dig, int64_t pitch, hipStream_t s);
hipError_t launch_weighted_csr_count(int64_t rows, int64_t t, int64_t* row_ptr, hipStream_t s);
hipError_t launch_weighted_csr_fill(const RngArgs& r, int64_t rows, int64_t cols, const int64_t* row_ptr,
                                    int32_t* col_idx, uint32_t* values, hipStream_t s);

hipError_t launch_mfma_probe(int mode, int64_t iters, int32_t* out, int64_t* ops, hipStream_t s);

// count = #{(i, j) : a(i, j) != b(i, j)}, or != 0 when b is null; with
// clear_count false the entries are added to a count some earlier launch on
// the stream has cleared.
hipError_t launch_count_mismatches(const uint32_t* a, int64_t lda, const uint32_t* b, int64_t ldb, int64_t rows,
                                   int64_t cols, int64_t* count, hipStream_t s, bool clear_count = true);

// Ring product C = A B^T with an epilogue.
// EPI_ACCUM adds the product to c (c += A B^T over the ring): long inner
// dimensions are split into chunks that each fit the int32 accumulators.
enum EpilogueKind { EPI_STORE = 0, EPI_UNMASK = 1, EPI_ACCUM = 2 };

// Inner-dimension chunk of one launch: the four-product shift class
// accumulates 4 K 2^14 < 2^31 only for K < 2^15; a multiple of 64.
constexpr int64_t MAX_K_CHUNK = 32704;
struct GemmLaunch {
  const int8_t* a;
  int64_t a_pitch;
  const int8_t* b;
  int64_t b_pitch;
  int64_t M, N, Kp;       // Kp: K padded to 64
  // B given as ring words: bytes of B's last row that may be read from
  // b (its valid words from b on, rounded up to 16 bytes)
  int64_t b_last;
  // A given as ring words (unmask of at most 16 rows): bytes of A's last
  // row that may be read (its K valid words)
  int64_t a_last;
  // decode kernel, EPI_ACCUM: subtract the product from c instead of adding
  bool negate;
  // tiled kernel (set by its launcher): the last split_tiles tiles run as
  // split_k pieces of the inner dimension, added into c atomically
  int64_t split_tiles;
  int32_t split_k;
  // EPI_STORE
  uint32_t* c;
  int64_t ldc;
  // EPI_UNMASK: out = ym - kc - acc (the elementwise unmask subtracts c,
  // when set, as a finished product)
  const uint32_t* ym;
  int64_t ldy;
  const uint32_t* kc;
  int64_t ldk;
  int32_t* y;
  int64_t ldo;
  const float* s_rows;
  const float* s_cols;
  const float* bias;      // optional, N entries, added to y_f32
  float* y_f32;
  int64_t ldf;
};
hipError_t launch_ring_gemm(const GemmLaunch& g, EpilogueKind epi, hipStream_t s);

// Products with at most SKINNY_MAX_M rows of A (decode shapes) run on a
// kernel that streams B once and splits K inside each workgroup.
constexpr int64_t SKINNY_MAX_M = 64;

// Compute units of the current device (cached per device id; host threads
// may call it concurrently).
inline int compute_units() {
  static std::atomic<int> cached[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) dev = 0;
  if (dev >= 0 && dev < 64) {
    const int c = cached[dev].load(std::memory_order_relaxed);
    if (c > 0) return c;
  }
  int v = 0;
  if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || v <= 0) v = 256;
  if (dev >= 0 && dev < 64) cached[dev].store(v, std::memory_order_relaxed);
  return v;
}
hipError_t launch_ring_gemm_skinny(const GemmLaunch& g, EpilogueKind epi, hipStream_t s);
// C = A B^T for A of at most SKINNY_MAX_M rows (digits) and B given as ring
// words (b = first word, b_pitch = row pitch in bytes, a multiple of 16);
// EPI_STORE or EPI_ACCUM.
hipError_t launch_ring_gemm_words_b(const GemmLaunch& g, EpilogueKind epi, hipStream_t s);
// Unmask (EPI_UNMASK) of at most 16 rows with A given as ring words (a,
// a_pitch bytes per row, a_last as above): the rows' digit planes are formed
// in registers as A is loaded.
hipError_t launch_unmask_words_a(const GemmLaunch& g, hipStream_t s);
// d = 0 (rows x cols, leading dimension ldd) and *count = 0 in one launch.
hipError_t launch_clear_check(uint32_t* d, int64_t ldd, int64_t rows, int64_t cols, int64_t* count, hipStream_t s);

// Writes one recombined ring value of C = A B^T at (m, n) through the
// epilogue: EPI_STORE stores it; EPI_UNMASK forms y = ym - val - kc and
// stores it as int32 and/or dequantised fp32 (plus the bias, added after the
// two scale products with no fused multiply-add).
template <int EPI>
__device__ __forceinline__ void gemm_epilogue(const GemmLaunch& g, int64_t m, int64_t n, uint32_t val) {
  if (EPI == EPI_STORE) {
    g.c[m * g.ldc + n] = val;
  } else if (EPI == EPI_ACCUM) {
    g.c[m * g.ldc + n] += val;
  } else {
    uint32_t y = g.ym[m * g.ldy + n] - val;
    if (g.kc != nullptr) y -= g.kc[m * g.ldk + n];
    if (g.y != nullptr) g.y[m * g.ldo + n] = (int32_t)y;
    if (g.y_f32 != nullptr) {
      const float v = (float)(int32_t)y * g.s_rows[m] * g.s_cols[n];
      g.y_f32[m * g.ldf + n] = g.bias != nullptr ? __fadd_rn(v, g.bias[n]) : v;
    }
  }
}

// True if the tile epilogue may use 16-byte accesses for every operand:
// N % 4 == 0 (so a 4-column chunk is wholly inside or outside the matrix),
// 16-byte aligned base pointers and row pitches that are multiples of 4.
inline bool gemm_epilogue_vectorizable(const GemmLaunch& g, EpilogueKind epi) {
  auto ok = [](const void* p, int64_t ld) { return p == nullptr || ((((uintptr_t)p) & 15) == 0 && (ld & 3) == 0); };
  if (g.N % 4 != 0) return false;
  if (epi == EPI_STORE || epi == EPI_ACCUM) return ok(g.c, g.ldc);
  return ok(g.ym, g.ldy) && ok(g.kc, g.ldk) && ok(g.y, g.ldo) && ok(g.y_f32, g.ldf) &&
         (g.y_f32 == nullptr || ((((uintptr_t)g.s_cols) & 15) == 0 && (((uintptr_t)g.bias) & 15) == 0));
}

// Epilogue of a TM x TN output tile held in LDS (row pitch TROW words) by a
// workgroup of NT threads: chunks of 4 consecutive columns, thread t taking
// chunks t, t + NT, .... VEC (see gemm_epilogue_vectorizable): 16-byte
// accesses, and the unmask inputs of all of a thread's chunks are loaded
// first, from addresses clamped into the matrix so that the loads need no
// branches (values of chunks outside the matrix are discarded). Otherwise one
// word at a time through gemm_epilogue.
template <int EPI, int VEC, int TM, int TN, int NT, int TROW>
__device__ __forceinline__ void gemm_tile_epilogue(const GemmLaunch& g, const uint32_t* tile, int64_t m0,
                                                   int64_t n0, int tid) {
  constexpr int CPR = TN / 4;                     // chunks per tile row
  constexpr int PER = TM * CPR / NT;              // chunks per thread
  static_assert(TM * CPR % NT == 0, "tile must split evenly");
  if (!VEC) {
    for (int k = 0; k < PER; ++k) {
      const int c = tid + NT * k;
      const int r = c / CPR;
      const int64_t m = m0 + r;
      const int64_t n = n0 + 4 * (c % CPR);
      for (int e = 0; e < 4; ++e)
        if (m < g.M && n + e < g.N) gemm_epilogue<EPI>(g, m, n + e, tile[r * TROW + 4 * (c % CPR) + e]);
    }
    return;
  }
  if (EPI == EPI_STORE) {
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int c = tid + NT * k;
      const int r = c / CPR;
      const int64_t m = m0 + r;
      const int64_t n = n0 + 4 * (c % CPR);
      if (m < g.M && n < g.N)
        *(uint4*)(g.c + m * g.ldc + n) = *(const uint4*)(tile + r * TROW + 4 * (c % CPR));
    }
    return;
  }
  if (EPI == EPI_ACCUM) {
    uint4 cv[PER];                                  // every c chunk is read before the first store
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int c = tid + NT * k;
      const int64_t m = min(m0 + c / CPR, g.M - 1);
      const int64_t n = min(n0 + 4 * (c % CPR), g.N - 4);
      cv[k] = *(const uint4*)(g.c + m * g.ldc + n);
    }
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int c = tid + NT * k;
      const int r = c / CPR;
      const int64_t m = m0 + r;
      const int64_t n = n0 + 4 * (c % CPR);
      if (m >= g.M || n >= g.N) continue;
      const uint4 a = *(const uint4*)(tile + r * TROW + 4 * (c % CPR));
      *(uint4*)(g.c + m * g.ldc + n) = make_uint4(cv[k].x + a.x, cv[k].y + a.y, cv[k].z + a.z, cv[k].w + a.w);
    }
    return;
  }
  const bool dq = g.y_f32 != nullptr;
  uint4 ymv[PER], kcv[PER];
  float4 scv[PER], bv[PER];
  float srv[PER];
#pragma unroll
  for (int k = 0; k < PER; ++k) {
    const int c = tid + NT * k;
    const int64_t m = min(m0 + c / CPR, g.M - 1);
    const int64_t n = min(n0 + 4 * (c % CPR), g.N - 4);
    ymv[k] = *(const uint4*)(g.ym + m * g.ldy + n);
    kcv[k] = g.kc != nullptr ? *(const uint4*)(g.kc + m * g.ldk + n) : make_uint4(0u, 0u, 0u, 0u);
    if (dq) {
      scv[k] = *(const float4*)(g.s_cols + n);
      srv[k] = g.s_rows[m];
      bv[k] = g.bias != nullptr ? *(const float4*)(g.bias + n) : make_float4(0.f, 0.f, 0.f, 0.f);
    }
  }
#pragma unroll
  for (int k = 0; k < PER; ++k) {
    const int c = tid + NT * k;
    const int r = c / CPR;
    const int64_t m = m0 + r;
    const int64_t n = n0 + 4 * (c % CPR);
    if (m >= g.M || n >= g.N) continue;
    const uint4 a = *(const uint4*)(tile + r * TROW + 4 * (c % CPR));
    const uint32_t o0 = ymv[k].x - kcv[k].x - a.x, o1 = ymv[k].y - kcv[k].y - a.y;
    const uint32_t o2 = ymv[k].z - kcv[k].z - a.z, o3 = ymv[k].w - kcv[k].w - a.w;
    if (g.y != nullptr) *(int4*)(g.y + m * g.ldo + n) = make_int4((int)o0, (int)o1, (int)o2, (int)o3);
    if (dq) {
      float4 f = make_float4((float)(int32_t)o0 * srv[k] * scv[k].x, (float)(int32_t)o1 * srv[k] * scv[k].y,
                             (float)(int32_t)o2 * srv[k] * scv[k].z, (float)(int32_t)o3 * srv[k] * scv[k].w);
      if (g.bias != nullptr)
        f = make_float4(__fadd_rn(f.x, bv[k].x), __fadd_rn(f.y, bv[k].y), __fadd_rn(f.z, bv[k].z),
                        __fadd_rn(f.w, bv[k].w));
      *(float4*)(g.y_f32 + m * g.ldf + n) = f;
    }
  }
}

// Unmask without a product term (R = 0): out = ym - kc.
hipError_t launch_unmask_elementwise(const GemmLaunch& g, hipStream_t s);

hipError_t launch_hadamard(const float* x, int64_t ldx, float* y, int64_t ldy, int64_t rows,
                           int64_t n, int log2_block, const int8_t* signs, int inverse,
                           hipStream_t s);
bool hadamard28_supported(int log2_block);
hipError_t launch_hadamard28(const float* x, int64_t ldx, float* y, int64_t ldy, int64_t rows, int log2_block,
                             const int8_t* signs, int inverse, hipStream_t s);

// Fused rotate + quantise + mask of Pi_Sec-Linear's input (secure_input.hip).
bool rotate_quantize_mask_supported(int log2_block);
hipError_t launch_rotate_quantize_mask(const float* x, int64_t ldx, int64_t rows, int64_t n, int log2_block,
                                       const int8_t* signs, int32_t qmax, const uint32_t* u, int64_t ldu,
                                       const RngArgs* noise, int8_t* out_dig, int64_t pitch, float* scale,
                                       hipStream_t s);

hipError_t launch_quantize_rows(const float* x, int64_t ldx, int64_t rows, int64_t n, int32_t qmax,
                                int32_t* q, int64_t ldq, int8_t* q_dig, int64_t q_pitch,
                                float* scale, hipStream_t s);

}  // namespace mosaic
