// Measurement aid: the rate of v_mfma_i32_32x32x32_i8 with operands held in
// registers (no memory traffic), for zero, constant and uniformly random
// operands. The ring product's kernels run the same instruction on uniform
// digits (masked operands are uniform by construction), so the random-operand
// rate is the ceiling those kernels work under.
#include "internal.h"

namespace mosaic {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));

__device__ __forceinline__ uint32_t mix(uint32_t x) {
  x ^= x >> 16;
  x *= 0x7FEB352Du;
  x ^= x >> 15;
  x *= 0x846CA68Bu;
  x ^= x >> 16;
  return x;
}

// MODE 0: zero operands; 1: the same constant operands for every MFMA;
// 2: four random operand sets per side, cycled so that both operands change
// from one MFMA to the next. Eight independent accumulators per wave.
template <int MODE>
__global__ __launch_bounds__(256) void mfma_probe_kernel(int64_t iters, uint32_t seed, int32_t* out) {
  v4i a[4], b[4];
  for (int j = 0; j < 4; ++j)
    for (int e = 0; e < 4; ++e) {
      const uint32_t t = (blockIdx.x * 256u + threadIdx.x) * 64u + (uint32_t)(j * 8 + e);
      a[j][e] = MODE == 0 ? 0 : MODE == 1 ? (int)(0x01020304u + (uint32_t)e) : (int)mix(2u * t + seed);
      b[j][e] = MODE == 0 ? 0 : MODE == 1 ? (int)(0x05060708u + (uint32_t)e) : (int)mix(2u * t + 1u + seed);
    }
  for (int j = 0; j < 4; ++j) asm volatile("" : "+v"(a[j]), "+v"(b[j]));
  v16i acc[8];
  for (int j = 0; j < 8; ++j)
    for (int v = 0; v < 16; ++v) acc[j][v] = 0;
#pragma unroll 1
  for (int64_t it = 0; it < iters; ++it) {
#pragma unroll
    for (int j = 0; j < 8; ++j)
      acc[j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a[j & 3], b[(j + (j >> 2)) & 3], acc[j], 0, 0, 0);
  }
  int s = 0;
  for (int j = 0; j < 8; ++j)
    for (int v = 0; v < 16; ++v) s += acc[j][v];
  atomicAdd(out, s);   // keeps the loop live; the value is not meaningful
}

}  // namespace

hipError_t launch_mfma_probe(int mode, int64_t iters, int32_t* out, int64_t* ops, hipStream_t s) {
  const int grid = 2 * compute_units();
  *ops = (int64_t)grid * 4 * iters * 8 * (2LL * 32 * 32 * 32);
  if (mode == 0) hipLaunchKernelGGL(mfma_probe_kernel<0>, dim3(grid), dim3(256), 0, s, iters, 1u, out);
  else if (mode == 1) hipLaunchKernelGGL(mfma_probe_kernel<1>, dim3(grid), dim3(256), 0, s, iters, 1u, out);
  else hipLaunchKernelGGL(mfma_probe_kernel<2>, dim3(grid), dim3(256), 0, s, iters, 1u, out);
  return hipGetLastError();
}

}  // namespace mosaic
