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

// Fast path for rows of a multiple of 4 elements with 16-byte aligned rows:
// thread c handles columns 4 c .. 4 c + 3 with one float4 load, so every
// load and store instruction of a wave covers one contiguous KiB. Pass 1
// reduces max |x| over the row (wave shuffles, then one LDS word per wave);
// pass 2 re-reads the row (now in L2), divides by the fp32 scale, rounds half
// to even and stores int32 codes with int4 stores and/or digit planes: the
// four lanes of a quad hold one 16-column group, and a quad shuffle hands
// each lane one 16-byte plane to store. Padding columns up to the next
// multiple of 64 get zero digits.
__global__ __launch_bounds__(256) void quantize_rows_vec_kernel(const float* __restrict__ x, int64_t ldx,
                                                                int64_t n, int32_t qmax, int32_t* q, int64_t ldq,
                                                                int8_t* q_dig, int64_t q_pitch, float* scale) {
  __shared__ float red[4];
  const int64_t row = blockIdx.x;
  const float4* xr = (const float4*)(x + row * ldx);
  const int64_t nv = n / 4;
  float m = 0.0f;
  for (int64_t c = threadIdx.x; c < nv; c += 256) {
    const float4 f = xr[c];
    m = fmaxf(m, fmaxf(fmaxf(fabsf(f.x), fabsf(f.y)), fmaxf(fabsf(f.z), fabsf(f.w))));
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) m = fmaxf(m, __shfl_xor(m, off));
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = m;
  __syncthreads();
  const float amax = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  const float s = (amax > 0.0f) ? amax / (float)qmax : 1.0f;
  if (threadIdx.x == 0 && scale != nullptr) scale[row] = s;

  const int64_t nchunks = q_dig ? 16 * ((n + 63) / 64) : nv;   // a multiple of 4 with digits
  for (int64_t c = threadIdx.x; c < nchunks; c += 256) {        // quads stay together (256 % 4 == 0)
    uint32_t v[4] = {0u, 0u, 0u, 0u};
    if (c < nv) {
      const float4 f = xr[c];
      v[0] = (uint32_t)(int32_t)rintf(f.x / s);
      v[1] = (uint32_t)(int32_t)rintf(f.y / s);
      v[2] = (uint32_t)(int32_t)rintf(f.z / s);
      v[3] = (uint32_t)(int32_t)rintf(f.w / s);
      if (q != nullptr)
        *(int4*)(q + row * ldq + 4 * c) = make_int4((int)v[0], (int)v[1], (int)v[2], (int)v[3]);
    }
    if (q_dig != nullptr) {
      uint32_t o[4];
      quad_digit_planes(v, (int)(c & 3), o);
      *(uint4*)(q_dig + row * q_pitch + 16 * c) = make_uint4(o[0], o[1], o[2], o[3]);
    }
  }
}

// Rows of at most 4 NT NV elements: the row is read once, with non-temporal
// loads, and kept in registers (thread t holds columns 4 (t + NT k) .. + 3,
// k < NV) between the max reduction and the code pass; stores are
// non-temporal. Same arithmetic and output layout as the kernels above.
template <int NT, int NV>
__global__ __launch_bounds__(NT) void quantize_rows_reg_kernel(const float* __restrict__ x, int64_t ldx,
                                                               int64_t n, int32_t qmax, int32_t* q, int64_t ldq,
                                                               int8_t* q_dig, int64_t q_pitch, float* scale) {
  constexpr int NW = NT / 64;
  __shared__ float red[NW];
  const int t = threadIdx.x;
  const int64_t row = blockIdx.x;
  const f32x4* xr = (const f32x4*)(x + row * ldx);
  const int64_t nv = n / 4;
  f32x4 f[NV];
#pragma unroll
  for (int k = 0; k < NV; ++k) {
    const int64_t c = t + NT * k;
    f[k] = c < nv ? __builtin_nontemporal_load(xr + c) : f32x4{0.0f, 0.0f, 0.0f, 0.0f};
  }
  float m = 0.0f;
#pragma unroll
  for (int k = 0; k < NV; ++k)
    m = fmaxf(m, fmaxf(fmaxf(fabsf(f[k][0]), fabsf(f[k][1])), fmaxf(fabsf(f[k][2]), fabsf(f[k][3]))));
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) m = fmaxf(m, __shfl_xor(m, off));
  if ((t & 63) == 0) red[t >> 6] = m;
  __syncthreads();
  float amax = red[0];
#pragma unroll
  for (int w = 1; w < NW; ++w) amax = fmaxf(amax, red[w]);
  const float s = (amax > 0.0f) ? amax / (float)qmax : 1.0f;
  if (t == 0 && scale != nullptr) scale[row] = s;

  const int64_t nchunks = q_dig ? 16 * ((n + 63) / 64) : nv;   // <= NT NV; a multiple of 4 with digits
#pragma unroll
  for (int k = 0; k < NV; ++k) {
    const int64_t c = t + NT * k;
    if (c >= nchunks) break;                                     // uniform per quad (NT % 4 == 0)
    uint32_t v[4] = {0u, 0u, 0u, 0u};
    if (c < nv) {
#pragma unroll
      for (int i = 0; i < 4; ++i) v[i] = (uint32_t)(int32_t)rintf(f[k][i] / s);
      if (q != nullptr) {
        const u32x4 ov = {v[0], v[1], v[2], v[3]};
        __builtin_nontemporal_store(ov, (u32x4*)(q + row * ldq + 4 * c));
      }
    }
    if (q_dig != nullptr) {
      uint32_t o[4];
      quad_digit_planes(v, (int)(c & 3), o);
      const u32x4 ov = {o[0], o[1], o[2], o[3]};
      __builtin_nontemporal_store(ov, (u32x4*)(q_dig + row * q_pitch + 16 * c));
    }
  }
}

template <int NT, int NV>
void launch_quantize_reg(const float* x, int64_t ldx, int64_t rows, int64_t n, int32_t qmax, int32_t* q,
                         int64_t ldq, int8_t* q_dig, int64_t q_pitch, float* scale, hipStream_t s) {
  hipLaunchKernelGGL((quantize_rows_reg_kernel<NT, NV>), dim3((unsigned)rows), dim3(NT), 0, s, x, ldx, n, qmax, q,
                     ldq, q_dig, q_pitch, scale);
}

}  // namespace

hipError_t launch_quantize_rows(const float* x, int64_t ldx, int64_t rows, int64_t n, int32_t qmax, int32_t* q,
                                int64_t ldq, int8_t* q_dig, int64_t q_pitch, float* scale, hipStream_t s) {
  if (rows == 0) return hipSuccess;
  const bool vec = n % 4 == 0 && ldx % 4 == 0 && ((uintptr_t)x & 15) == 0 &&
                   (q == nullptr || (ldq % 4 == 0 && ((uintptr_t)q & 15) == 0)) &&
                   (q_dig == nullptr || ((uintptr_t)q_dig & 15) == 0);
  // register-resident rows: 256 threads up to n = 16384, 1024 threads up to 65536
  if (vec && n <= 1024) launch_quantize_reg<256, 1>(x, ldx, rows, n, qmax, q, ldq, q_dig, q_pitch, scale, s);
  else if (vec && n <= 2048) launch_quantize_reg<256, 2>(x, ldx, rows, n, qmax, q, ldq, q_dig, q_pitch, scale, s);
  else if (vec && n <= 4096) launch_quantize_reg<256, 4>(x, ldx, rows, n, qmax, q, ldq, q_dig, q_pitch, scale, s);
  else if (vec && n <= 8192) launch_quantize_reg<256, 8>(x, ldx, rows, n, qmax, q, ldq, q_dig, q_pitch, scale, s);
  else if (vec && n <= 16384) launch_quantize_reg<256, 16>(x, ldx, rows, n, qmax, q, ldq, q_dig, q_pitch, scale, s);
  else if (vec && n <= 32768) launch_quantize_reg<1024, 8>(x, ldx, rows, n, qmax, q, ldq, q_dig, q_pitch, scale, s);
  else if (vec && n <= 65536) launch_quantize_reg<1024, 16>(x, ldx, rows, n, qmax, q, ldq, q_dig, q_pitch, scale, s);
  else if (vec)
    hipLaunchKernelGGL(quantize_rows_vec_kernel, dim3((unsigned)rows), dim3(256), 0, s, x, ldx, n, qmax, q, ldq,
                       q_dig, q_pitch, scale);
  else
    hipLaunchKernelGGL(quantize_rows_kernel, dim3((unsigned)rows), dim3(256), 0, s, x, ldx, n, qmax, q, ldq,
                       q_dig, q_pitch, scale);
  return hipGetLastError();
}

}  // namespace mosaic
