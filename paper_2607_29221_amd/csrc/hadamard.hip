// Random Hadamard rotation (Section 5): per block of b = 2^LOGB consecutive
// elements of a row, forward y = H_b (d * x) / sqrt(b), inverse
// y = d * (H_b x) / sqrt(b), with H_b in Sylvester order. One workgroup per
// block: the block transform of fwht_block.h, then the scale (and, for the
// inverse, the signs) and coalesced 16-byte stores. The whole block stays in
// LDS (b <= 32768 floats = 128 KiB), so HBM sees one read and one write per
// element.
#include "fwht_block.h"

namespace mosaic {
namespace {

// SIGNS: 0 none, 1 applied on load (forward), 2 applied on store (inverse).
// x is read once and y written once, so both use non-temporal accesses.
template <int LOGB, int SIGNS>
__global__ __launch_bounds__((FwhtShape<LOGB, fwht_tmax(LOGB)>::T)) void fwht_kernel(
    const float* __restrict__ x, int64_t ldx, float* y, int64_t ldy, int64_t blocks_per_row,
    const int8_t* __restrict__ signs, float scale) {
  constexpr int TM = fwht_tmax(LOGB);
  using S = FwhtShape<LOGB, TM>;
  constexpr int T = S::T, E = S::E, NV = S::NV, B = S::B;
  __shared__ float sm[S::SM];
  const int t = threadIdx.x;
  const int64_t row = blockIdx.x / blocks_per_row;
  const int64_t blk = blockIdx.x - row * blocks_per_row;
  const float* xr = x + row * ldx + blk * B;
  float* yr = y + row * ldy + blk * B;
  const int8_t* sg = SIGNS ? signs + blk * B : nullptr;

  float v[E];
  fwht_load<LOGB, SIGNS == 1, true, TM>(xr, sg, v);
  const float sc = scale * fwht_transform<LOGB, TM>(sm, v);   // the transform's lane sign folded into the scale
#pragma unroll
  for (int r = 0; r < E; ++r) v[r] *= sc;
  if (SIGNS == 2) apply_signs<LOGB, TM>(sg, v);
#pragma unroll
  for (int k = 0; k < NV; ++k) {
    const f32x4 f = {v[4 * k], v[4 * k + 1], v[4 * k + 2], v[4 * k + 3]};
    __builtin_nontemporal_store(f, (f32x4*)yr + t + T * k);
  }
}

template <int LOGB>
hipError_t launch_fwht(const float* x, int64_t ldx, float* y, int64_t ldy, int64_t rows, int64_t n,
                       const int8_t* signs, int inverse, hipStream_t s) {
  constexpr int B = FwhtShape<LOGB, fwht_tmax(LOGB)>::B;
  constexpr int T = FwhtShape<LOGB, fwht_tmax(LOGB)>::T;
  const int64_t bpr = n / B;
  const int64_t grid = rows * bpr;
  if (grid == 0) return hipSuccess;
  const float scale = (float)(1.0 / sqrt((double)B));
  if (signs == nullptr)
    hipLaunchKernelGGL((fwht_kernel<LOGB, 0>), dim3((unsigned)grid), dim3(T), 0, s, x, ldx, y, ldy, bpr, signs,
                       scale);
  else if (!inverse)
    hipLaunchKernelGGL((fwht_kernel<LOGB, 1>), dim3((unsigned)grid), dim3(T), 0, s, x, ldx, y, ldy, bpr, signs,
                       scale);
  else
    hipLaunchKernelGGL((fwht_kernel<LOGB, 2>), dim3((unsigned)grid), dim3(T), 0, s, x, ldx, y, ldy, bpr, signs,
                       scale);
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
