// Per-row fixed-point quantisation of Pi_Sec-Linear (Section 5 protocol box):
// s = max |row| / qmax (1 for an all-zero row), q = round-half-even(x / s),
// both in fp32 with correctly rounded division. One block per row: a max
// reduction, then one thread per 16-column group writes the codes as int32
// and/or in the digit layout (sign-extended into the ring, zero padding).
#include "internal.h"

namespace mosaic {
namespace {

__global__ __launch_bounds__(256) void quantize_rows_kernel(const float* __restrict__ x, int64_t ldx,
                                                            int64_t n, int32_t qmax, int32_t* q, int64_t ldq,
                                                            int8_t* q_dig, int64_t q_pitch, float* scale) {
  __shared__ float red[256];
  const int64_t row = blockIdx.x;
  const float* xr = x + row * ldx;
  float m = 0.0f;
  for (int64_t j = threadIdx.x; j < n; j += blockDim.x) m = fmaxf(m, fabsf(xr[j]));
  red[threadIdx.x] = m;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) red[threadIdx.x] = fmaxf(red[threadIdx.x], red[threadIdx.x + w]);
    __syncthreads();
  }
  const float amax = red[0];
  const float s = (amax > 0.0f) ? amax / (float)qmax : 1.0f;
  if (threadIdx.x == 0 && scale != nullptr) scale[row] = s;

  const int64_t groups = q_dig ? (64 * ((n + 63) / 64)) / 16 : (n + 15) / 16;
  for (int64_t g = threadIdx.x; g < groups; g += blockDim.x) {
    int32_t c[16];
#pragma unroll
    for (int b = 0; b < 16; ++b) {
      const int64_t j = 16 * g + b;
      c[b] = (j < n) ? (int32_t)rintf(xr[j] / s) : 0;
    }
    if (q != nullptr) {
      for (int b = 0; b < 16; ++b)
        if (16 * g + b < n) q[row * ldq + 16 * g + b] = c[b];
    }
    if (q_dig != nullptr) {
      uint32_t planes[4][4];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const uint32_t w[4] = {digit_word((uint32_t)c[4 * k]), digit_word((uint32_t)c[4 * k + 1]),
                               digit_word((uint32_t)c[4 * k + 2]), digit_word((uint32_t)c[4 * k + 3])};
        uint32_t t4[4];
        digit_transpose4(w, t4);
#pragma unroll
        for (int t = 0; t < 4; ++t) planes[t][k] = t4[t];
      }
      uint4* dp = (uint4*)(q_dig + row * q_pitch + 64 * g);
#pragma unroll
      for (int t = 0; t < 4; ++t) dp[t] = make_uint4(planes[t][0], planes[t][1], planes[t][2], planes[t][3]);
    }
  }
}

}  // namespace

hipError_t launch_quantize_rows(const float* x, int64_t ldx, int64_t rows, int64_t n, int32_t qmax, int32_t* q,
                                int64_t ldq, int8_t* q_dig, int64_t q_pitch, float* scale, hipStream_t s) {
  if (rows == 0) return hipSuccess;
  hipLaunchKernelGGL(quantize_rows_kernel, dim3((unsigned)rows), dim3(256), 0, s, x, ldx, n, qmax, q, ldq,
                     q_dig, q_pitch, scale);
  return hipGetLastError();
}

}  // namespace mosaic
