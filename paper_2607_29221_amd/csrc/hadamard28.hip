// Rotation by H_28 (x) H_b for rows of n = 28 b entries (Section 5's random
// Hadamard rotation for a length that is not a power of two, e.g. the
// 28672 = 28 x 1024 feed-forward width): entry i b + j of a row is entry j of
// block i, and the rotation mixes every entry of the row, where the
// block-diagonal I_28 (x) H_b mixes only within blocks.
//
//   forward:  y = (H_28 (x) H_b) (d * x) / sqrt(n)
//   inverse:  y = d * ((H_28^T (x) H_b) x) / sqrt(n)   (the transpose)
//
// H_28 is Paley's first construction over GF(27) = GF(3)[t] / (t^3 + 2t + 1):
// H = I + S, S = [[0, 1^T], [-1, Q]], Q[i][k] = chi(e_i - e_k), chi the
// quadratic character and e_i the field element with base-3 digits of i as
// coefficients of 1, t, t^2. Since 27 = 3 (mod 4), S is skew-symmetric and
// H H^T = 28 I. The table is built at compile time below.
//
// One workgroup of b / 4 threads per row. Thread t holds columns 4 t .. 4 t + 3
// of all 28 blocks (112 floats): per block, exactly the register layout of
// the block transform in fwht_block.h (b = 2^LOGB, 4 elements per thread), so
// H_b runs through that transform, seven blocks per LDS pass; H_28 then mixes the 28
// blocks of each column in registers, through the sums below (its +-1
// entries folded into adds). HBM traffic: one read and one write per element.
#include "fwht_block.h"

namespace mosaic {
namespace {

constexpr int gf27_mul(int a, int b) {
  int pa[3] = {a % 3, (a / 3) % 3, a / 9};
  int pb[3] = {b % 3, (b / 3) % 3, b / 9};
  int pr[5] = {0, 0, 0, 0, 0};
  for (int i = 0; i < 3; ++i)
    for (int j = 0; j < 3; ++j) pr[i + j] += pa[i] * pb[j];
  // t^3 = t + 2 (mod t^3 + 2t + 1 over GF(3)); reduce t^4, then t^3
  for (int k = 4; k >= 3; --k) {
    const int c = pr[k];
    pr[k] = 0;
    pr[k - 2] += c;
    pr[k - 3] += 2 * c;
  }
  return pr[0] % 3 + 3 * (pr[1] % 3) + 9 * (pr[2] % 3);
}

constexpr int gf27_sub(int a, int b) {
  const int c0 = ((a % 3) - (b % 3) + 3) % 3;
  const int c1 = (((a / 3) % 3) - ((b / 3) % 3) + 3) % 3;
  const int c2 = ((a / 9) - (b / 9) + 3) % 3;
  return c0 + 3 * c1 + 9 * c2;
}

struct Paley28 {
  signed char h[28][28];
};

constexpr Paley28 make_paley28() {
  bool square[27] = {};
  for (int a = 1; a < 27; ++a) square[gf27_mul(a, a)] = true;
  Paley28 p{};
  for (int i = 0; i < 28; ++i)
    for (int k = 0; k < 28; ++k) {
      int s = 0;                                            // S[i][k]
      if (i == 0 && k > 0) s = 1;
      else if (i > 0 && k == 0) s = -1;
      else if (i > 0 && k > 0) {
        const int e = gf27_sub(i - 1, k - 1);
        s = e == 0 ? 0 : (square[e] ? 1 : -1);
      }
      p.h[i][k] = (signed char)(s + (i == k ? 1 : 0));
    }
  return p;
}

constexpr Paley28 kH28 = make_paley28();

constexpr bool paley28_is_hadamard() {
  for (int i = 0; i < 28; ++i)
    for (int k = 0; k < 28; ++k) {
      int dot = 0;
      for (int j = 0; j < 28; ++j) dot += kH28.h[i][j] * kH28.h[k][j];
      if (dot != (i == k ? 28 : 0)) return false;
    }
  return true;
}
static_assert(paley28_is_hadamard(), "H_28 must satisfy H H^T = 28 I");

// SIGNS: 0 none, 1 on load (forward), 2 on store (inverse). INV selects H_28^T.
template <int LOGB, int SIGNS, bool INV>
__global__ __launch_bounds__(FwhtShape<LOGB>::T) void fwht28_kernel(const float* __restrict__ x, int64_t ldx,
                                                                      float* y, int64_t ldy,
                                                                      const int8_t* __restrict__ signs, float scale) {
  using S = FwhtShape<LOGB>;
  constexpr int T = S::T, B = S::B;
  static_assert(S::E == 4, "one float4 per thread and block");
  constexpr int G = 7;                    // blocks per shared LDS pass of the block transform
  __shared__ float sm[G * S::SM];
  const int t = threadIdx.x;
  const int64_t row = blockIdx.x;
  const float* xr = x + row * ldx;
  float* yr = y + row * ldy;

  float v[28][4];
#pragma unroll
  for (int i = 0; i < 28; ++i) {
    const f32x4 f = __builtin_nontemporal_load((const f32x4*)(xr + i * B) + t);
    v[i][0] = f[0]; v[i][1] = f[1]; v[i][2] = f[2]; v[i][3] = f[3];
  }
  if (SIGNS == 1) {
#pragma unroll
    for (int i = 0; i < 28; ++i) apply_signs<LOGB>(signs + i * B, v[i]);
  }
  float c = 1.0f;
#pragma unroll
  for (int g = 0; g < 28; g += G) {
    c = fwht_transform_blocks<LOGB, G>(sm, reinterpret_cast<float (&)[G][4]>(v[g]));   // same lane sign
    __syncthreads();                       // the next group reuses the scratch
  }
  // H_28 across the blocks, column by column. With H = I + S, T = sum of
  // v_1 .. v_27, U = v_0 + T and P_i the sum of the 13 v_k (k >= 1, k != i)
  // with Q[i-1][k-1] = +1 (so that row i of Q v is 2 P_i - T + v_i):
  //   H v:    y_0 = U,      y_i = 2 (v_i + P_i) - U
  //   H^T v:  y_0 = v_0 - T, y_i = U - 2 P_i          (S^T = -S)
  // 405 adds per column instead of 784.
  const float sc = scale * c;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    float tsum = v[1][q];
#pragma unroll
    for (int k = 2; k < 28; ++k) tsum += v[k][q];
    const float u = v[0][q] + tsum;
    float o[28];
    o[0] = INV ? v[0][q] - tsum : u;
#pragma unroll
    for (int i = 1; i < 28; ++i) {
      float pi = INV ? 0.0f : v[i][q];
#pragma unroll
      for (int k = 1; k < 28; ++k)
        if (k != i && kH28.h[i][k] > 0) pi += v[k][q];
      o[i] = INV ? __builtin_fmaf(-2.0f, pi, u) : __builtin_fmaf(2.0f, pi, -u);
    }
#pragma unroll
    for (int i = 0; i < 28; ++i) v[i][q] = o[i] * sc;
  }
  if (SIGNS == 2) {
#pragma unroll
    for (int i = 0; i < 28; ++i) apply_signs<LOGB>(signs + i * B, v[i]);
  }
#pragma unroll
  for (int i = 0; i < 28; ++i) {
    const f32x4 f = {v[i][0], v[i][1], v[i][2], v[i][3]};
    __builtin_nontemporal_store(f, (f32x4*)(yr + i * B) + t);
  }
}

template <int LOGB>
hipError_t launch_fwht28(const float* x, int64_t ldx, float* y, int64_t ldy, int64_t rows, const int8_t* signs,
                         int inverse, hipStream_t s) {
  using S = FwhtShape<LOGB>;
  const float scale = (float)(1.0 / sqrt(28.0 * (double)S::B));
  const dim3 grid((unsigned)rows), block(S::T);
  if (signs == nullptr && !inverse)
    hipLaunchKernelGGL((fwht28_kernel<LOGB, 0, false>), grid, block, 0, s, x, ldx, y, ldy, signs, scale);
  else if (signs == nullptr)
    hipLaunchKernelGGL((fwht28_kernel<LOGB, 0, true>), grid, block, 0, s, x, ldx, y, ldy, signs, scale);
  else if (!inverse)
    hipLaunchKernelGGL((fwht28_kernel<LOGB, 1, false>), grid, block, 0, s, x, ldx, y, ldy, signs, scale);
  else
    hipLaunchKernelGGL((fwht28_kernel<LOGB, 2, true>), grid, block, 0, s, x, ldx, y, ldy, signs, scale);
  return hipGetLastError();
}

}  // namespace

bool hadamard28_supported(int log2_block) { return log2_block >= 8 && log2_block <= 10; }

hipError_t launch_hadamard28(const float* x, int64_t ldx, float* y, int64_t ldy, int64_t rows, int log2_block,
                             const int8_t* signs, int inverse, hipStream_t s) {
  if (rows == 0) return hipSuccess;
  switch (log2_block) {
    case 8: return launch_fwht28<8>(x, ldx, y, ldy, rows, signs, inverse, s);
    case 9: return launch_fwht28<9>(x, ldx, y, ldy, rows, signs, inverse, s);
    case 10: return launch_fwht28<10>(x, ldx, y, ldy, rows, signs, inverse, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace mosaic
