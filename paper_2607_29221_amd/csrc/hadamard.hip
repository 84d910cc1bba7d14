// Random Hadamard rotation (Section 5): per block of b = 2^LOGB consecutive
// elements of a row, forward y = H_b (d * x) / sqrt(b), inverse
// y = d * (H_b x) / sqrt(b), with H_b in Sylvester order applied by Fino's
// butterflies (a, b) -> (a + b, a - b), one stage per index bit.
//
// The butterfly stages on different index bits commute, so the kernel does
// them in the order the data layout makes cheap:
//  * each thread loads E = b / T elements as float4s at positions
//    4 (t + T k) + q -- coalesced 16-byte loads across the block -- and runs
//    the stages on the bits it holds in registers (bits 0-1 from q and the
//    top bits from k);
//  * the remaining middle bits 2 .. 2 + log2 T - 1 cross threads: the row goes
//    to LDS and each pass gathers 2^e elements that differ in e consecutive
//    middle bits, runs those stages in registers and writes them back;
//  * the row is read back in the load layout, scaled (and signed, for the
//    inverse) and stored with coalesced 16-byte stores.
// LDS addresses are padded by one word per 32 (idx + idx / 32), which makes
// the strided gathers conflict-free. The whole block stays in LDS
// (b <= 32768 floats = 128 KiB), so HBM sees one read and one write per
// element.
#include "internal.h"

namespace mosaic {
namespace {

__host__ __device__ constexpr int ilog2c(int v) { return v <= 1 ? 0 : 1 + ilog2c(v >> 1); }

__device__ __forceinline__ int pad(int idx) { return idx + (idx >> 5); }

template <int LOGB>
__global__ __launch_bounds__(((1 << LOGB) / 4 < 256) ? (1 << LOGB) / 4 : 256) void fwht_kernel(
    const float* __restrict__ x, int64_t ldx, float* y, int64_t ldy, int64_t blocks_per_row,
    const int8_t* __restrict__ signs, int inverse, float scale) {
  constexpr int B = 1 << LOGB;
  constexpr int T = (B / 4 < 256) ? B / 4 : 256;
  constexpr int LOGT = ilog2c(T);
  constexpr int E = B / T;            // elements per thread, >= 4
  constexpr int LOGE = LOGB - LOGT;
  constexpr int NV = E / 4;
  __shared__ float sm[B + B / 32];

  const int t = threadIdx.x;
  const int64_t row = blockIdx.x / blocks_per_row;
  const int64_t blk = blockIdx.x - row * blocks_per_row;
  const float* xr = x + row * ldx + blk * B;
  float* yr = y + row * ldy + blk * B;
  const int8_t* sg = signs ? signs + blk * B : nullptr;

  float v[E];
#pragma unroll
  for (int k = 0; k < NV; ++k) {
    const float4 f = ((const float4*)xr)[t + T * k];
    v[4 * k + 0] = f.x; v[4 * k + 1] = f.y; v[4 * k + 2] = f.z; v[4 * k + 3] = f.w;
    if (!inverse && sg) {
      const char4 s4 = ((const char4*)sg)[t + T * k];
      v[4 * k + 0] *= (float)s4.x; v[4 * k + 1] *= (float)s4.y;
      v[4 * k + 2] *= (float)s4.z; v[4 * k + 3] *= (float)s4.w;
    }
  }

  // stages on the index bits held in registers: bits of r = 4 k + q
#pragma unroll
  for (int h = 1; h < E; h <<= 1) {
#pragma unroll
    for (int r = 0; r < E; ++r) {
      if ((r & h) == 0) {
        const float a = v[r], b = v[r + h];
        v[r] = a + b;
        v[r + h] = a - b;
      }
    }
  }

  if (LOGT > 0) {
#pragma unroll
    for (int r = 0; r < E; ++r) sm[pad(4 * (t + T * (r >> 2)) + (r & 3))] = v[r];
    __syncthreads();

    // middle bits [2, 2 + LOGT), LOGE at a time
#pragma unroll
    for (int p = 2; p < 2 + LOGT; p += LOGE) {
      const int e = (2 + LOGT - p) < LOGE ? (2 + LOGT - p) : LOGE;
      const int n_in = 1 << e;
      const int groups = E / n_in;
      for (int gi = 0; gi < groups; ++gi) {
        const int o = t + T * gi;
        const int low = o & ((1 << p) - 1);
        const int high = o >> p;
        const int base = low | (high << (p + e));
        float w[E];
#pragma unroll
        for (int i = 0; i < E; ++i)
          if (i < n_in) w[i] = sm[pad(base | (i << p))];
#pragma unroll
        for (int h = 1; h < E; h <<= 1) {
          if (h < n_in) {
#pragma unroll
            for (int i = 0; i < E; ++i) {
              if (i < n_in && (i & h) == 0) {
                const float a = w[i], b = w[i + h];
                w[i] = a + b;
                w[i + h] = a - b;
              }
            }
          }
        }
#pragma unroll
        for (int i = 0; i < E; ++i)
          if (i < n_in) sm[pad(base | (i << p))] = w[i];
      }
      __syncthreads();
    }

#pragma unroll
    for (int r = 0; r < E; ++r) v[r] = sm[pad(4 * (t + T * (r >> 2)) + (r & 3))];
  }

#pragma unroll
  for (int k = 0; k < NV; ++k) {
    float4 f = make_float4(v[4 * k] * scale, v[4 * k + 1] * scale, v[4 * k + 2] * scale, v[4 * k + 3] * scale);
    if (inverse && sg) {
      const char4 s4 = ((const char4*)sg)[t + T * k];
      f.x *= (float)s4.x; f.y *= (float)s4.y; f.z *= (float)s4.z; f.w *= (float)s4.w;
    }
    ((float4*)yr)[t + T * k] = f;
  }
}

template <int LOGB>
hipError_t launch_fwht(const float* x, int64_t ldx, float* y, int64_t ldy, int64_t rows, int64_t n,
                       const int8_t* signs, int inverse, hipStream_t s) {
  constexpr int B = 1 << LOGB;
  constexpr int T = (B / 4 < 256) ? B / 4 : 256;
  const int64_t bpr = n / B;
  const int64_t grid = rows * bpr;
  if (grid == 0) return hipSuccess;
  const float scale = (float)(1.0 / sqrt((double)B));
  hipLaunchKernelGGL(fwht_kernel<LOGB>, dim3((unsigned)grid), dim3(T), 0, s, x, ldx, y, ldy, bpr, signs,
                     inverse, scale);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_hadamard(const float* x, int64_t ldx, float* y, int64_t ldy, int64_t rows, int64_t n,
                           int log2_block, const int8_t* signs, int inverse, hipStream_t s) {
  switch (log2_block) {
    case 4: return launch_fwht<4>(x, ldx, y, ldy, rows, n, signs, inverse, s);
    case 5: return launch_fwht<5>(x, ldx, y, ldy, rows, n, signs, inverse, s);
    case 6: return launch_fwht<6>(x, ldx, y, ldy, rows, n, signs, inverse, s);
    case 7: return launch_fwht<7>(x, ldx, y, ldy, rows, n, signs, inverse, s);
    case 8: return launch_fwht<8>(x, ldx, y, ldy, rows, n, signs, inverse, s);
    case 9: return launch_fwht<9>(x, ldx, y, ldy, rows, n, signs, inverse, s);
    case 10: return launch_fwht<10>(x, ldx, y, ldy, rows, n, signs, inverse, s);
    case 11: return launch_fwht<11>(x, ldx, y, ldy, rows, n, signs, inverse, s);
    case 12: return launch_fwht<12>(x, ldx, y, ldy, rows, n, signs, inverse, s);
    case 13: return launch_fwht<13>(x, ldx, y, ldy, rows, n, signs, inverse, s);
    case 14: return launch_fwht<14>(x, ldx, y, ldy, rows, n, signs, inverse, s);
    case 15: return launch_fwht<15>(x, ldx, y, ldy, rows, n, signs, inverse, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace mosaic
