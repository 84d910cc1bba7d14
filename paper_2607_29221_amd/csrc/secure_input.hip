// Client input pass of Pi_Sec-Linear (Section 5 protocol box, online step 1,
// followed by the mask of the Section 4.2 protocol box, online step 2) fused
// into one kernel: for every token row x (n floats)
//   1. rotate blockwise, y = H_b (d * x) / sqrt(b)   (b = 2^LOGB, n = k b);
//   2. quantise, s = max_j |y_j| / q_max (1 for an all-zero row),
//      q_j = round-half-even(y_j / s);
//   3. mask, A'_j = q_j + U_j + E_j over Z_{2^32}, E drawn in the pass;
//   4. write A' as digits, and s.
// It performs exactly the arithmetic of mosaic_hadamard_rotate,
// mosaic_quantize_rows and mosaic_mask in sequence (same butterfly order,
// same fp32 scale, the same correctly rounded quotient before rounding to an
// integer, same noise element indices), so the digits are bit-identical to
// that sequence, with 16 bytes of HBM traffic per element instead of 28 for
// the three passes. The pass is bound by vector-ALU issue, so the quotient
// of each code is replaced by a product with the reciprocal of the scale
// wherever that provably rounds to the same integer (quant_codes4).
//
// Rows that fit in registers with room to spare (n = 8192 with b = 8192,
// 4096 or 1024, and 16384 with b = 16384) run in one launch
// (rqm_row_kernel: 12 bytes per element; 8-28% faster than two launches
// there). A 28672-float row held whole needs about 180 registers per lane:
// the few workgroups that fit made it 47% slower, so it takes the two
// launches. Otherwise two launches, one
// workgroup per row each, with only the block transform's scratch in LDS
// (so occupancy is that of the plain rotation): the first
// rotates the row block by block and keeps only max |y| (written to
// scale[row]); the second rotates again -- the butterflies are cheap next to
// the memory traffic -- quantises with s = max / q_max, adds u and the noise
// and writes the digits, then replaces scale[row] by s. HBM traffic: x twice,
// u once, digits once (16 bytes per element).
#include "fwht_block.h"

namespace mosaic {
namespace {

// The block shape of the rotation kernel for the same b (same butterfly order).
template <int LOGB>
using FS = FwhtShape<LOGB, fwht_tmax(LOGB)>;

template <int LOGB>
__device__ __forceinline__ float block_max(float m, float* red) {
  constexpr int T = FS<LOGB>::T;
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) m = fmaxf(m, __shfl_xor(m, off));
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = m;
  __syncthreads();
  float r = red[0];
#pragma unroll
  for (int w = 1; w < T / 64; ++w) r = fmaxf(r, red[w]);
  return r;
}

template <int LOGB, bool SG>
__global__ __launch_bounds__((FS<LOGB>::T)) void rqm_max_kernel(const float* __restrict__ x, int64_t ldx,
                                                                     int64_t n, const int8_t* __restrict__ signs,
                                                                     float scale_b, float* amax_out) {
  using S = FS<LOGB>;
  constexpr int E = S::E, B = S::B;
  static_assert(S::T % 256 == 0, "full waves on every SIMD");
  __shared__ float sm[S::SM];
  __shared__ float red[S::T / 64];
  const int64_t row = blockIdx.x;
  const float* xr = x + row * ldx;
  float m = 0.0f;
  for (int64_t blk = 0; blk < n / B; ++blk) {
    float v[E];
    // x is read again by the next launch: cached loads
    fwht_load<LOGB, SG, false, fwht_tmax(LOGB)>(xr + blk * B, SG ? signs + blk * B : nullptr, v);
    fwht_transform<LOGB, fwht_tmax(LOGB)>(sm, v);    // the lane sign it returns does not change |y|
#pragma unroll
    for (int r = 0; r < E; ++r) m = fmaxf(m, fabsf(v[r] * scale_b));
    __syncthreads();                // the next block reuses the scratch
  }
  const float amax = block_max<LOGB>(m, red);
  if (threadIdx.x == 0) amax_out[row] = amax;
}

// SG, HU, HN: signs, u and noise present (compile-time, so that no run-time
// test sits between a load and its use). Each 16-byte word of u is requested
// where it is used: requesting a block's words ahead (before the transform,
// or all before the first use) holds them in registers, fewer workgroups fit
// and the pass ran 10-25% slower.
template <int LOGB, bool SG, bool HU, bool HN>
__global__ __launch_bounds__((FS<LOGB>::T), (FS<LOGB>::WAVES)) void rqm_mask_kernel(
    const float* __restrict__ x, int64_t ldx, int64_t n, const int8_t* __restrict__ signs, float scale_b,
    int32_t qmax, const uint32_t* __restrict__ u, int64_t ldu, RngArgs noise, int8_t* out_dig, int64_t pitch,
    float* scale) {
  using S = FS<LOGB>;
  constexpr int T = S::T, E = S::E, NV = S::NV, B = S::B;
  __shared__ float sm[S::SM];
  const int t = threadIdx.x;
  const int64_t row = blockIdx.x;
  const float* xr = x + row * ldx;
  const float amax = scale[row];    // written by rqm_max_kernel
  const float s = (amax > 0.0f) ? amax / (float)qmax : 1.0f;
  const float rs = 1.0f / s, thr = quant_threshold(s, qmax);
  for (int64_t blk = 0; blk < n / B; ++blk) {
    float v[E];
    fwht_load<LOGB, SG, true, fwht_tmax(LOGB)>(xr + blk * B, SG ? signs + blk * B : nullptr, v);
    const float sb = scale_b * fwht_transform<LOGB, fwht_tmax(LOGB)>(sm, v);   // the lane sign folded into the scale
    const float kb = sb * rs;
#pragma unroll
    for (int k = 0; k < NV; ++k) {
      // columns 4 c .. 4 c + 3 of the row; lanes t .. t + 3 hold one 16-column group
      const int64_t c = blk * (B / 4) + t + T * k;
      const u32x4 uu = HU ? __builtin_nontemporal_load((const u32x4*)(u + row * ldu + 4 * c)) : u32x4{0, 0, 0, 0};
      uint32_t w[4];
      quant_codes4(&v[4 * k], sb, kb, s, thr, w);
      w[0] += uu[0]; w[1] += uu[1]; w[2] += uu[2]; w[3] += uu[3];
      if (HN) {
        uint32_t e[4];
        sample4_aligned(noise, (uint64_t)row * (uint64_t)n + (uint64_t)(4 * c), e);
        w[0] += e[0]; w[1] += e[1]; w[2] += e[2]; w[3] += e[3];
      }
      uint32_t o[4];
      quad_digit_planes(w, t & 3, o);
      const u32x4 ov = {o[0], o[1], o[2], o[3]};
      __builtin_nontemporal_store(ov, (u32x4*)(out_dig + row * pitch + 16 * c));
    }
    __syncthreads();                // the next block reuses the scratch
  }
  if (t == 0) scale[row] = s;       // every thread read the maximum before the first barrier
}

// Rows held whole in registers (NB blocks of b = 2^LOGB, NB E floats per
// thread): one launch. Each thread loads its share of the row once, the
// blocks are rotated G per LDS pass, max |y| is reduced across the workgroup,
// and the codes are formed, masked and written from the same registers:
// 12 bytes of HBM traffic per element instead of 16, the same arithmetic as
// the two launches above (so the same digits). Signs and u are present.
template <int LOGB, int NB, int G, bool HN>
__global__ __launch_bounds__((FS<LOGB>::T)) void rqm_row_kernel(
    const float* __restrict__ x, int64_t ldx, const int8_t* __restrict__ signs, float scale_b, int32_t qmax,
    const uint32_t* __restrict__ u, int64_t ldu, RngArgs noise, int8_t* out_dig, int64_t pitch, float* scale) {
  using S = FS<LOGB>;
  constexpr int T = S::T, E = S::E, NV = S::NV, B = S::B;
  constexpr int64_t n = (int64_t)NB * B;
  static_assert(NB % G == 0, "groups of G blocks");
  __shared__ float sm[G * S::SM];
  __shared__ float red[T / 64];
  const int t = threadIdx.x;
  const int64_t row = blockIdx.x;
  const float* xr = x + row * ldx;

  float v[NB][E];
#pragma unroll
  for (int k = 0; k < NB; ++k) fwht_load<LOGB, true, true, fwht_tmax(LOGB)>(xr + k * B, signs + k * B, v[k]);
  float c = 1.0f;
#pragma unroll
  for (int g = 0; g < NB; g += G) {
    // every group returns the same lane sign
    c = fwht_transform_blocks<LOGB, G, fwht_tmax(LOGB)>(sm, reinterpret_cast<float (&)[G][E]>(v[g]));
    __syncthreads();
  }
  float m = 0.0f;
#pragma unroll
  for (int k = 0; k < NB; ++k)
#pragma unroll
    for (int r = 0; r < E; ++r) m = fmaxf(m, fabsf(v[k][r] * scale_b));
  const float amax = block_max<LOGB>(m, red);
  const float s = (amax > 0.0f) ? amax / (float)qmax : 1.0f;
  const float sb = scale_b * c;
  const float kb = sb * (1.0f / s), thr = quant_threshold(s, qmax);
#pragma unroll
  for (int k = 0; k < NB; ++k) {
#pragma unroll
    for (int kk = 0; kk < NV; ++kk) {
      // columns 4 cc .. 4 cc + 3 of the row; lanes t .. t + 3 hold one 16-column group
      const int64_t cc = k * (B / 4) + t + T * kk;
      const u32x4 uu = __builtin_nontemporal_load((const u32x4*)(u + row * ldu + 4 * cc));
      uint32_t w[4];
      quant_codes4(&v[k][4 * kk], sb, kb, s, thr, w);
      w[0] += uu[0]; w[1] += uu[1]; w[2] += uu[2]; w[3] += uu[3];
      if (HN) {
        uint32_t e[4];
        sample4_aligned(noise, (uint64_t)row * (uint64_t)n + (uint64_t)(4 * cc), e);
        w[0] += e[0]; w[1] += e[1]; w[2] += e[2]; w[3] += e[3];
      }
      uint32_t o[4];
      quad_digit_planes(w, t & 3, o);
      const u32x4 ov = {o[0], o[1], o[2], o[3]};
      __builtin_nontemporal_store(ov, (u32x4*)(out_dig + row * pitch + 16 * cc));
    }
  }
  if (t == 0) scale[row] = s;
}

template <int LOGB, int NB, int G>
hipError_t launch_rqm_row(const float* x, int64_t ldx, int64_t rows, const int8_t* signs, int32_t qmax,
                          const uint32_t* u, int64_t ldu, const RngArgs* noise, int8_t* out_dig, int64_t pitch,
                          float* scale, hipStream_t s) {
  using S = FS<LOGB>;
  const float scale_b = (float)(1.0 / sqrt((double)S::B));
  if (noise != nullptr)
    hipLaunchKernelGGL((rqm_row_kernel<LOGB, NB, G, true>), dim3((unsigned)rows), dim3(S::T), 0, s, x, ldx, signs,
                       scale_b, qmax, u, ldu, *noise, out_dig, pitch, scale);
  else
    hipLaunchKernelGGL((rqm_row_kernel<LOGB, NB, G, false>), dim3((unsigned)rows), dim3(S::T), 0, s, x, ldx,
                       signs, scale_b, qmax, u, ldu, RngArgs{}, out_dig, pitch, scale);
  return hipGetLastError();
}

template <int LOGB, bool SG, bool HU, bool HN>
hipError_t launch_rqm_t(const float* x, int64_t ldx, int64_t rows, int64_t n, const int8_t* signs, int32_t qmax,
                        const uint32_t* u, int64_t ldu, const RngArgs* noise, int8_t* out_dig, int64_t pitch,
                        float* scale, hipStream_t s) {
  using S = FS<LOGB>;
  const float scale_b = (float)(1.0 / sqrt((double)S::B));
  hipLaunchKernelGGL((rqm_max_kernel<LOGB, SG>), dim3((unsigned)rows), dim3(S::T), 0, s, x, ldx, n, signs, scale_b,
                     scale);
  hipLaunchKernelGGL((rqm_mask_kernel<LOGB, SG, HU, HN>), dim3((unsigned)rows), dim3(S::T), 0, s, x, ldx, n, signs,
                     scale_b, qmax, u, ldu, HN ? *noise : RngArgs{}, out_dig, pitch, scale);
  return hipGetLastError();
}

template <int LOGB, bool SG, bool HU>
hipError_t launch_rqm_n(const float* x, int64_t ldx, int64_t rows, int64_t n, const int8_t* signs, int32_t qmax,
                        const uint32_t* u, int64_t ldu, const RngArgs* noise, int8_t* out_dig, int64_t pitch,
                        float* scale, hipStream_t s) {
  if (noise != nullptr)
    return launch_rqm_t<LOGB, SG, HU, true>(x, ldx, rows, n, signs, qmax, u, ldu, noise, out_dig, pitch, scale, s);
  return launch_rqm_t<LOGB, SG, HU, false>(x, ldx, rows, n, signs, qmax, u, ldu, noise, out_dig, pitch, scale, s);
}

template <int LOGB, bool SG>
hipError_t launch_rqm_u(const float* x, int64_t ldx, int64_t rows, int64_t n, const int8_t* signs, int32_t qmax,
                        const uint32_t* u, int64_t ldu, const RngArgs* noise, int8_t* out_dig, int64_t pitch,
                        float* scale, hipStream_t s) {
  if (u != nullptr)
    return launch_rqm_n<LOGB, SG, true>(x, ldx, rows, n, signs, qmax, u, ldu, noise, out_dig, pitch, scale, s);
  return launch_rqm_n<LOGB, SG, false>(x, ldx, rows, n, signs, qmax, u, ldu, noise, out_dig, pitch, scale, s);
}

template <int LOGB>
hipError_t launch_rqm(const float* x, int64_t ldx, int64_t rows, int64_t n, const int8_t* signs, int32_t qmax,
                      const uint32_t* u, int64_t ldu, const RngArgs* noise, int8_t* out_dig, int64_t pitch,
                      float* scale, hipStream_t s) {
  if (signs != nullptr)
    return launch_rqm_u<LOGB, true>(x, ldx, rows, n, signs, qmax, u, ldu, noise, out_dig, pitch, scale, s);
  return launch_rqm_u<LOGB, false>(x, ldx, rows, n, signs, qmax, u, ldu, noise, out_dig, pitch, scale, s);
}

}  // namespace

bool rotate_quantize_mask_supported(int log2_block) { return log2_block >= 10 && log2_block <= 14; }

hipError_t launch_rotate_quantize_mask(const float* x, int64_t ldx, int64_t rows, int64_t n, int log2_block,
                                       const int8_t* signs, int32_t qmax, const uint32_t* u, int64_t ldu,
                                       const RngArgs* noise, int8_t* out_dig, int64_t pitch, float* scale,
                                       hipStream_t s) {
  if (rows == 0) return hipSuccess;
  if (signs != nullptr && u != nullptr) {
    // rows that fit in registers: one launch
    const int64_t nb = n >> log2_block;
    if (log2_block == 13 && nb == 1)
      return launch_rqm_row<13, 1, 1>(x, ldx, rows, signs, qmax, u, ldu, noise, out_dig, pitch, scale, s);
    if (log2_block == 12 && nb == 2)
      return launch_rqm_row<12, 2, 2>(x, ldx, rows, signs, qmax, u, ldu, noise, out_dig, pitch, scale, s);
    if (log2_block == 10 && nb == 8)
      return launch_rqm_row<10, 8, 4>(x, ldx, rows, signs, qmax, u, ldu, noise, out_dig, pitch, scale, s);
    if (log2_block == 14 && nb == 1)
      return launch_rqm_row<14, 1, 1>(x, ldx, rows, signs, qmax, u, ldu, noise, out_dig, pitch, scale, s);
  }
  switch (log2_block) {
    case 10: return launch_rqm<10>(x, ldx, rows, n, signs, qmax, u, ldu, noise, out_dig, pitch, scale, s);
    case 11: return launch_rqm<11>(x, ldx, rows, n, signs, qmax, u, ldu, noise, out_dig, pitch, scale, s);
    case 12: return launch_rqm<12>(x, ldx, rows, n, signs, qmax, u, ldu, noise, out_dig, pitch, scale, s);
    case 13: return launch_rqm<13>(x, ldx, rows, n, signs, qmax, u, ldu, noise, out_dig, pitch, scale, s);
    case 14: return launch_rqm<14>(x, ldx, rows, n, signs, qmax, u, ldu, noise, out_dig, pitch, scale, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace mosaic
