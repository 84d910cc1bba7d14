// Launch interfaces between the C ABI layer (abi.cpp) and the kernel files.
// Every launcher assumes its arguments were validated by the ABI layer.
#pragma once

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

// Ring product C = A B^T with an epilogue.
enum EpilogueKind { EPI_STORE = 0, EPI_UNMASK = 1 };
struct GemmLaunch {
  const int8_t* a;
  int64_t a_pitch;
  const int8_t* b;
  int64_t b_pitch;
  int64_t M, N, Kp;       // Kp: K padded to 64
  // EPI_STORE
  uint32_t* c;
  int64_t ldc;
  // EPI_UNMASK: out = ym - kc - acc
  const uint32_t* ym;
  int64_t ldy;
  const uint32_t* kc;
  int64_t ldk;
  int32_t* y;
  int64_t ldo;
  const float* s_rows;
  const float* s_cols;
  float* y_f32;
  int64_t ldf;
};
hipError_t launch_ring_gemm(const GemmLaunch& g, EpilogueKind epi, hipStream_t s);

// Products with at most SKINNY_MAX_M rows of A (decode shapes) run on a
// kernel that streams B once and splits K inside each workgroup.
constexpr int64_t SKINNY_MAX_M = 64;
hipError_t launch_ring_gemm_skinny(const GemmLaunch& g, EpilogueKind epi, hipStream_t s);

// Writes one recombined ring value of C = A B^T at (m, n) through the
// epilogue: EPI_STORE stores it; EPI_UNMASK forms y = ym - val - kc and
// stores it as int32 and/or dequantised fp32.
template <int EPI>
__device__ __forceinline__ void gemm_epilogue(const GemmLaunch& g, int64_t m, int64_t n, uint32_t val) {
  if (EPI == EPI_STORE) {
    g.c[m * g.ldc + n] = val;
  } else {
    uint32_t y = g.ym[m * g.ldy + n] - val;
    if (g.kc != nullptr) y -= g.kc[m * g.ldk + n];
    if (g.y != nullptr) g.y[m * g.ldo + n] = (int32_t)y;
    if (g.y_f32 != nullptr) g.y_f32[m * g.ldf + n] = (float)(int32_t)y * g.s_rows[m] * g.s_cols[n];
  }
}

// Unmask without a product term (R = 0): out = ym - kc.
hipError_t launch_unmask_elementwise(const GemmLaunch& g, hipStream_t s);

hipError_t launch_hadamard(const float* x, int64_t ldx, float* y, int64_t ldy, int64_t rows,
                           int64_t n, int log2_block, const int8_t* signs, int inverse,
                           hipStream_t s);

hipError_t launch_quantize_rows(const float* x, int64_t ldx, int64_t rows, int64_t n, int32_t qmax,
                                int32_t* q, int64_t ldq, int8_t* q_dig, int64_t q_pitch,
                                float* scale, hipStream_t s);

}  // namespace mosaic
