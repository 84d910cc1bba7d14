// Walsh-Hadamard block transform shared by the rotation kernel and the fused
// rotate-quantise-mask kernel: Fino's butterflies (a, b) -> (a + b, a - b)
// over one block of b = 2^LOGB consecutive floats, Sylvester order. The
// stages on different index bits commute, so they run in the order the data
// layout makes cheap:
//  * each of the T threads loads E = b / T elements as float4s at positions
//    4 (t + T k) + q -- coalesced 16-byte loads across the block -- and runs
//    the stages on the bits it holds in registers (bits 0-1 from q and the
//    top bits from k);
//  * the stages on index bits 2-7, the lane bits of t, exchange values
//    between the lanes of a wave (DPP, swizzle and lane-swap instructions);
//  * the stages on the wave bits of t (index bits 8 .. 1 + log2 T: 8-9 for
//    256 threads, 8-10 for 512; present for b >= 512) go
//    through LDS in one pass: the block is written out, each thread gathers
//    2, 4 or 8 elements that differ in those bits, runs the stages and writes
//    them back, and the result is read back in the load layout (register r
//    of thread t holds element 4 (t + T (r / 4)) + r % 4), unscaled.
// LDS addresses are padded by one word per 32 (idx + idx / 32), which makes
// the strided gathers conflict-free.
#pragma once

#include "internal.h"

namespace mosaic {

__host__ __device__ constexpr int ilog2c(int v) { return v <= 1 ? 0 : 1 + ilog2c(v >> 1); }

// TMAX: most threads per block transform (256, or 512 for kernels that want
// more waves per block).
template <int LOGB, int TMAX = 256>
struct FwhtShape {
  static constexpr int B = 1 << LOGB;
  static constexpr int T = (B / 4 < TMAX) ? B / 4 : TMAX;  // threads per block transform
  static constexpr int LOGT = ilog2c(T);
  static constexpr int E = B / T;                           // elements per thread, >= 4
  static constexpr int LOGE = LOGB - LOGT;
  static constexpr int NV = E / 4;
  static constexpr int SM = B + B / 32;                     // LDS floats (padded)
  // workgroups of T threads that fit one CU's 160 KiB of LDS, as waves per
  // SIMD (T = 256: one wave per SIMD per workgroup), capped at 4; used as the
  // occupancy the register allocation must allow
  static constexpr int LDS_WG = (160 * 1024) / (SM * 4);
  static constexpr int WG_W = T >= 256 ? T / 256 : 1;     // waves per SIMD of one workgroup
  static constexpr int WAVES = T < 256 ? 4 : (LDS_WG * WG_W < 4 ? (LDS_WG < 1 ? WG_W : LDS_WG * WG_W) : 4);
};

// Threads per block transform in the rotation kernel and the fused input
// kernels (they must agree: the thread count fixes which butterfly stages
// run in registers, lanes or LDS, and so the rounding). 512 for b = 8192,
// where the block's LDS (33 KiB) admits four workgroups per compute unit:
// eight waves per workgroup instead of four double the waves resident and
// halve each thread's share of the block (4096 x 8192 rotation: 45.3 against
// 47.0 us); 256 otherwise.
__host__ __device__ constexpr int fwht_tmax(int logb) { return logb == 13 ? 512 : 256; }

// One thread's share of a block, as registers.
template <int LOGB, int TMAX = 256>
using FwhtRegs = float[FwhtShape<LOGB, TMAX>::E];

__device__ __forceinline__ int fwht_pad(int idx) { return idx + (idx >> 5); }

// v[r] *= d of its element (load layout), d = +-1 from the int8 signs at sg.
template <int LOGB, int TMAX = 256>
__device__ __forceinline__ void apply_signs(const int8_t* __restrict__ sg, FwhtRegs<LOGB, TMAX>& v) {
  using S = FwhtShape<LOGB, TMAX>;
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
template <int LOGB, bool SG, bool NT, int TMAX = 256>
__device__ __forceinline__ void fwht_load(const float* __restrict__ xr, const int8_t* __restrict__ sg,
                                          FwhtRegs<LOGB, TMAX>& v) {
  using S = FwhtShape<LOGB, TMAX>;
  constexpr int T = S::T, NV = S::NV;
  const int t = threadIdx.x;
#pragma unroll
  for (int k = 0; k < NV; ++k) {
    const f32x4* p = (const f32x4*)xr + t + T * k;
    const f32x4 f = NT ? __builtin_nontemporal_load(p) : *p;
    v[4 * k + 0] = f[0]; v[4 * k + 1] = f[1]; v[4 * k + 2] = f[2]; v[4 * k + 3] = f[3];
  }
  if (SG) apply_signs<LOGB, TMAX>(sg, v);
}

// Value of x held by lane (lane ^ M) of the wave, M in {1, 2, 4, 8}: DPP
// quad permutes for 1 and 2, a swizzle for 4, a DPP row rotation by 8
// (within 16 lanes) for 8.
template <int M>
__device__ __forceinline__ float lane_xor(float x) {
  const int xi = __float_as_int(x);
  int p;
  if constexpr (M == 1) {
    p = __builtin_amdgcn_mov_dpp(xi, 0xB1, 0xF, 0xF, false);          // quad_perm [1, 0, 3, 2]
  } else if constexpr (M == 2) {
    p = __builtin_amdgcn_mov_dpp(xi, 0x4E, 0xF, 0xF, false);          // quad_perm [2, 3, 0, 1]
  } else if constexpr (M == 4) {
    p = __builtin_amdgcn_ds_swizzle(xi, 0x1F | (4 << 10));            // lane ^ 4 within 32 lanes
  } else {
    static_assert(M == 8, "lane_xor: M in {1, 2, 4, 8}");
    p = __builtin_amdgcn_mov_dpp(xi, 0x128, 0xF, 0xF, false);         // row_ror:8
  }
  return __int_as_float(p);
}

// Butterfly stage on lane bit M (1, 2, 4 or 8) of every register, in one
// fused multiply-add per value: w + sgn * partner with sgn = -1 on the upper
// lane of each pair. The lower lane gets a + b; the upper gets b - a, the
// negated difference. Signs are tracked rather than fixed: after the stages
// on lane bits in a set S, a lane holds (-1)^popcount(lane & S) times the
// true value, and the two lanes of a later pair carry the same sign, so the
// recurrence holds stage after stage. Rounding to nearest is symmetric, so
// this is bit-exact with the plain sum and difference up to that sign.
template <int M, int E>
__device__ __forceinline__ void lane_stage(float (&v)[E], int lane) {
  const float sgn = (lane & M) ? -1.0f : 1.0f;
#pragma unroll
  for (int r = 0; r < E; ++r) v[r] = __builtin_fmaf(lane_xor<M>(v[r]), sgn, v[r]);
}

// Exchange of lane bit log2 M (M = 16 or 32) with register bit log2 H: for
// each pair of registers r, r + H (r without bit H), the gfx950 row-swap
// instruction trades the halves whose two bits differ, after which the
// element in register r' of lane l is the one that sat in lane l with bit M
// set to bit H of r', register r' with bit H set to bit M of l. An
// involution: applied twice it restores the layout.
template <int M, int H, int E>
__device__ __forceinline__ void lane_exchange(float (&v)[E]) {
  static_assert(M == 16 || M == 32, "lane_exchange: M in {16, 32}");
#pragma unroll
  for (int r = 0; r < E; ++r) {
    if (r & H) continue;
    const unsigned x = __float_as_uint(v[r]), y = __float_as_uint(v[r + H]);
    const auto sw = (M == 16) ? __builtin_amdgcn_permlane16_swap(x, y, false, false)
                              : __builtin_amdgcn_permlane32_swap(x, y, false, false);
    v[r] = __uint_as_float(sw[0]);
    v[r + H] = __uint_as_float(sw[1]);
  }
}

// Butterfly stage on register bit log2 H.
template <int H, int E>
__device__ __forceinline__ void reg_stage(float (&v)[E]) {
#pragma unroll
  for (int r = 0; r < E; ++r) {
    if (r & H) continue;
    const float a = v[r], b = v[r + H];
    v[r] = a + b;
    v[r + H] = a - b;
  }
}

// In-place unscaled H_b of a block held in the load layout, up to a sign per
// lane: returns c = +-1 such that the true result in every register of this
// thread is c * v[r] (callers fold c into the scale they apply anyway). Every
// thread of the workgroup (FwhtShape<LOGB>::T of them) must call it; sm must
// not be in use by other threads when it is called (it is untouched for
// b <= 256).
//
// Index bits of the element in register r of thread t (t = lane + 64 wave):
// bits 0-1 are r % 4, bits 2 .. 1 + log2 T are t, the rest are r / 4. The
// stages on register bits run in registers. Those on lane bits 0-3 (index
// bits 2-5) take the partner's value by DPP or swizzle; those on lane bits 4
// and 5 (index bits 6, 7) exchange the lane bit with register bit 1 or 0 by
// row swaps and run in registers. The stages on wave bits (index bits 8 ..
// 1 + log2 T, present for b >= 512) go through one LDS pass, whose write addresses
// undo the two exchanges; for b <= 256 the exchanges are swapped back.
// The stages that stay inside the wave (registers, lanes), for one block;
// returns the lane sign c. For b >= 512 the element layout is left with the
// two lane/register exchanges in place (the LDS pass undoes them).
template <int LOGB, int TMAX = 256>
__device__ __forceinline__ float fwht_in_wave(FwhtRegs<LOGB, TMAX>& v, int lane) {
  using S = FwhtShape<LOGB, TMAX>;
  constexpr int LOGT = S::LOGT, E = S::E;

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

  // lane bits 0-3
  if constexpr (LOGT > 0) lane_stage<1>(v, lane);
  if constexpr (LOGT > 1) lane_stage<2>(v, lane);
  if constexpr (LOGT > 2) lane_stage<4>(v, lane);
  if constexpr (LOGT > 3) lane_stage<8>(v, lane);
  constexpr int done = (1 << (LOGT < 4 ? LOGT : 4)) - 1;
  const float c = (__builtin_popcount(lane & done) & 1) ? -1.0f : 1.0f;

  // lane bits 4 and 5 (E >= 4 whenever T >= 32)
  if constexpr (LOGT > 4) {
    lane_exchange<16, 2>(v);
    reg_stage<2>(v);
  }
  if constexpr (LOGT > 5) {
    lane_exchange<32, 1>(v);
    reg_stage<1>(v);
  }
  if constexpr (LOGT <= 6) {
    if constexpr (LOGT > 5) lane_exchange<32, 1>(v);
    if constexpr (LOGT > 4) lane_exchange<16, 2>(v);
  }
  return c;
}

// In-place unscaled H_b of NB blocks held in the load layout (v[k] one block),
// up to a sign per lane: returns c = +-1 such that the true result in every
// register of this thread is c * v[k][r] (callers fold c into the scale they
// apply anyway). Every thread of the workgroup (FwhtShape<LOGB>::T of them)
// must call it; sm (NB x FwhtShape<LOGB>::SM floats) must not be in use by
// other threads when it is called (it is untouched for b <= 256). The NB
// blocks share the LDS pass, so its two barriers are paid once.
//
// Index bits of the element in register r of thread t (t = lane + 64 wave):
// bits 0-1 are r % 4, bits 2 .. 1 + log2 T are t, the rest are r / 4. The
// stages on register bits run in registers. Those on lane bits 0-3 (index
// bits 2-5) take the partner's value by DPP or swizzle; those on lane bits 4
// and 5 (index bits 6, 7) exchange the lane bit with register bit 1 or 0 by
// row swaps and run in registers. The stages on wave bits (index bits 8 ..
// 1 + log2 T, present for b >= 512) go through one LDS pass, whose write addresses
// undo the two exchanges; for b <= 256 the exchanges are swapped back.
template <int LOGB, int NB, int TMAX = 256>
__device__ __forceinline__ float fwht_transform_blocks(float* sm, FwhtRegs<LOGB, TMAX> (&v)[NB]) {
  using S = FwhtShape<LOGB, TMAX>;
  constexpr int T = S::T, LOGT = S::LOGT, E = S::E, SM = S::SM;
  const int t = threadIdx.x;
  const int lane = t & 63;
  float c = 1.0f;
#pragma unroll
  for (int k = 0; k < NB; ++k) c = fwht_in_wave<LOGB, TMAX>(v[k], lane);   // the same c for every block

  if constexpr (LOGT > 6) {
    // Write every element at its index: register r of lane l now holds the
    // element of lane (l & 15) + 16 bit1(r) + 32 bit0(r), register
    // (r & ~3) + bit5(l) + 2 bit4(l). The per-register part of the index is a
    // multiple of 64, so the padded address splits the same way.
    const int base = 4 * ((t & ~63) + (lane & 15)) + ((lane >> 5) & 1) + 2 * ((lane >> 4) & 1);
    const int pbase = fwht_pad(base);
#pragma unroll
    for (int k = 0; k < NB; ++k)
#pragma unroll
      for (int r = 0; r < E; ++r) {
        const int off = 64 * ((r >> 1) & 1) + 128 * (r & 1) + 4 * T * (r >> 2);
        sm[k * SM + pbase + off + (off >> 5)] = v[k][r];
      }
    __syncthreads();
    // wave bits [8, 2 + LOGT): one pass over groups of 2^e elements
    constexpr int p = 8, e = LOGT - 6, n_in = 1 << e, groups = E / n_in;
#pragma unroll
    for (int k = 0; k < NB; ++k) {
      for (int gi = 0; gi < groups; ++gi) {
        const int o = t + T * gi;
        const int low = o & ((1 << p) - 1);
        const int high = o >> p;
        const int gbase = low | (high << (p + e));
        float w[n_in];
#pragma unroll
        for (int i = 0; i < n_in; ++i) w[i] = sm[k * SM + fwht_pad(gbase | (i << p))];
#pragma unroll
        for (int h = 1; h < n_in; h <<= 1) {
#pragma unroll
          for (int i = 0; i < n_in; ++i) {
            if ((i & h) == 0) {
              const float a = w[i], b = w[i + h];
              w[i] = a + b;
              w[i + h] = a - b;
            }
          }
        }
#pragma unroll
        for (int i = 0; i < n_in; ++i) sm[k * SM + fwht_pad(gbase | (i << p))] = w[i];
      }
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < NB; ++k)
#pragma unroll
      for (int r = 0; r < E; ++r) v[k][r] = sm[k * SM + fwht_pad(4 * (t + T * (r >> 2)) + (r & 3))];
  }
  return c;
}

// One block (see fwht_transform_blocks).
template <int LOGB, int TMAX = 256>
__device__ __forceinline__ float fwht_transform(float* sm, FwhtRegs<LOGB, TMAX>& v) {
  return fwht_transform_blocks<LOGB, 1, TMAX>(sm, reinterpret_cast<FwhtRegs<LOGB, TMAX> (&)[1]>(v));
}

}  // namespace mosaic
