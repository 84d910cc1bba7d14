// Walsh-Hadamard block transform shared by the rotation kernel and the fused
// rotate-quantise-mask kernel: Fino's butterflies (a, b) -> (a + b, a - b)
// over one block of b = 2^LOGB consecutive floats, Sylvester order. The
// stages on different index bits commute, so they run in the order the data
// layout makes cheap:
//  * each of the T threads loads E = b / T elements as float4s at positions
//    4 (t + T k) + q -- coalesced 16-byte loads across the block -- and runs
//    the stages on the bits it holds in registers (bits 0-1 from q and the
//    top bits from k);
//  * the remaining middle bits 2 .. 2 + log2 T - 1 cross threads: the block
//    goes to LDS and each pass gathers 2^e elements that differ in e
//    consecutive middle bits, runs those stages in registers and writes them
//    back;
//  * the result is read back in the load layout (register r of thread t holds
//    element 4 (t + T (r / 4)) + r % 4), unscaled.
// LDS addresses are padded by one word per 32 (idx + idx / 32), which makes
// the strided gathers conflict-free.
#pragma once

#include "internal.h"

namespace mosaic {

__host__ __device__ constexpr int ilog2c(int v) { return v <= 1 ? 0 : 1 + ilog2c(v >> 1); }

template <int LOGB>
struct FwhtShape {
  static constexpr int B = 1 << LOGB;
  static constexpr int T = (B / 4 < 256) ? B / 4 : 256;   // threads per block transform
  static constexpr int LOGT = ilog2c(T);
  static constexpr int E = B / T;                           // elements per thread, >= 4
  static constexpr int LOGE = LOGB - LOGT;
  static constexpr int NV = E / 4;
  static constexpr int SM = B + B / 32;                     // LDS floats (padded)
};

__device__ __forceinline__ int fwht_pad(int idx) { return idx + (idx >> 5); }

// v[r] *= d of its element (load layout), d = +-1 from the int8 signs at sg.
template <int LOGB>
__device__ __forceinline__ void apply_signs(const int8_t* __restrict__ sg, float (&v)[FwhtShape<LOGB>::E]) {
  using S = FwhtShape<LOGB>;
  constexpr int T = S::T, NV = S::NV;
  const int t = threadIdx.x;
#pragma unroll
  for (int k = 0; k < NV; ++k) {
    const char4 s4 = ((const char4*)sg)[t + T * k];
    v[4 * k + 0] *= (float)s4.x; v[4 * k + 1] *= (float)s4.y;
    v[4 * k + 2] *= (float)s4.z; v[4 * k + 3] *= (float)s4.w;
  }
}

// This thread's share of the block at xr in the load layout (register r of
// thread t: element 4 (t + T (r / 4)) + r % 4), times the signs at sg if SG.
// NT selects non-temporal loads, for data that is read once. Signs are a
// compile-time choice: a run-time test between the loads serialises them.
template <int LOGB, bool SG, bool NT>
__device__ __forceinline__ void fwht_load(const float* __restrict__ xr, const int8_t* __restrict__ sg,
                                          float (&v)[FwhtShape<LOGB>::E]) {
  using S = FwhtShape<LOGB>;
  constexpr int T = S::T, NV = S::NV;
  const int t = threadIdx.x;
#pragma unroll
  for (int k = 0; k < NV; ++k) {
    const f32x4* p = (const f32x4*)xr + t + T * k;
    const f32x4 f = NT ? __builtin_nontemporal_load(p) : *p;
    v[4 * k + 0] = f[0]; v[4 * k + 1] = f[1]; v[4 * k + 2] = f[2]; v[4 * k + 3] = f[3];
  }
  if (SG) apply_signs<LOGB>(sg, v);
}

// In-place unscaled H_b of a block held in the load layout. Every thread of
// the workgroup (FwhtShape<LOGB>::T of them) must call it; sm must not be in
// use by other threads when it is called.
template <int LOGB>
__device__ __forceinline__ void fwht_transform(float* sm, float (&v)[FwhtShape<LOGB>::E]) {
  using S = FwhtShape<LOGB>;
  constexpr int T = S::T, LOGT = S::LOGT, E = S::E, LOGE = S::LOGE;
  const int t = threadIdx.x;

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
    for (int r = 0; r < E; ++r) sm[fwht_pad(4 * (t + T * (r >> 2)) + (r & 3))] = v[r];
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
          if (i < n_in) w[i] = sm[fwht_pad(base | (i << p))];
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
          if (i < n_in) sm[fwht_pad(base | (i << p))] = w[i];
      }
      __syncthreads();
    }

#pragma unroll
    for (int r = 0; r < E; ++r) v[r] = sm[fwht_pad(4 * (t + T * (r >> 2)) + (r & 3))];
  }
}

}  // namespace mosaic
