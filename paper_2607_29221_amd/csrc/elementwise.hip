// Elementwise passes of the MOSAIC path: the mask pass (x + u + e -> ring
// elements and/or digit layout), sampling (the same pass with only e), the
// rotation's sign vector, and unmasking without a product term.
//
// One thread owns one 16-column digit group of one row: it reads 16 plaintext
// values, 16 ring words of u, draws 16 noise values (four Philox blocks when
// the group starts on a block boundary), and writes the four 16-byte digit
// planes of the group -- contiguous 64-byte chunks, so a wave writes 4 KiB of
// consecutive memory.
#include "internal.h"

namespace mosaic {
namespace {

__device__ __forceinline__ uint32_t load_x(const void* x, int32_t dt, int64_t off) {
  switch (dt) {
    case 0: return (uint32_t)(int32_t)((const int8_t*)x)[off];
    case 1: return (uint32_t)(int32_t)((const int16_t*)x)[off];
    case 2: return (uint32_t)((const int32_t*)x)[off];
    default: return ((const uint32_t*)x)[off];
  }
}

__global__ __launch_bounds__(256) void mask_kernel(MaskLaunch a, int64_t groups) {
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t i = gid / groups;
  const int64_t g = gid - i * groups;
  if (i >= a.rows) return;
  const int64_t j0 = 16 * g;
  const bool full = (j0 + 16 <= a.cols);
  uint32_t v[16];

  // plaintext
  if (a.x != nullptr) {
    if (full && a.x_dtype == 0 && a.x_cs == 1 &&
        ((((uintptr_t)a.x) + i * a.x_rs + j0) & 15) == 0) {
      const uint4 w = *(const uint4*)((const int8_t*)a.x + i * a.x_rs + j0);
      const uint32_t ww[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
      for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int b = 0; b < 4; ++b) v[4 * q + b] = (uint32_t)(int32_t)(int8_t)(ww[q] >> (8 * b));
    } else {
#pragma unroll
      for (int b = 0; b < 16; ++b) {
        const int64_t j = j0 + b;
        v[b] = (j < a.cols) ? load_x(a.x, a.x_dtype, i * a.x_rs + j * a.x_cs) : 0u;
      }
    }
  } else {
#pragma unroll
    for (int b = 0; b < 16; ++b) v[b] = 0u;
  }

  // precomputed ring mask
  if (a.u != nullptr) {
    const uint32_t* up = a.u + i * a.ldu + j0;
    if (full && ((((uintptr_t)up) & 15) == 0)) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const uint4 w = ((const uint4*)up)[q];
        v[4 * q + 0] += w.x; v[4 * q + 1] += w.y; v[4 * q + 2] += w.z; v[4 * q + 3] += w.w;
      }
    } else {
#pragma unroll
      for (int b = 0; b < 16; ++b)
        if (j0 + b < a.cols) v[b] += up[b];
    }
  }

  // noise drawn in the pass
  if (a.has_noise) {
    const RngArgs& r = a.noise;
    if (!r.transposed) {
      const uint64_t e0 = (uint64_t)i * (uint64_t)a.cols + (uint64_t)j0;
      if (full && (e0 & 3) == 0) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          uint32_t e4[4];
          sample4_aligned(r, e0 + 4 * q, e4);
          v[4 * q + 0] += e4[0]; v[4 * q + 1] += e4[1]; v[4 * q + 2] += e4[2]; v[4 * q + 3] += e4[3];
        }
      } else {
        for (int b = 0; b < 16; ++b)
          if (j0 + b < a.cols) v[b] += sample_elem(r, e0 + b);
      }
    } else {
      // logical matrix is cols x rows; output (i, j) is its element (j, i)
      for (int b = 0; b < 16; ++b) {
        const int64_t j = j0 + b;
        if (j < a.cols) v[b] += sample_elem(r, (uint64_t)j * (uint64_t)a.rows + (uint64_t)i);
      }
    }
  }

  // padding columns of a digit group are zero
  if (!full) {
#pragma unroll
    for (int b = 0; b < 16; ++b)
      if (j0 + b >= a.cols) v[b] = 0u;
  }

  if (a.out != nullptr) {
    uint32_t* op = a.out + i * a.ldo + j0;
    if (full && ((((uintptr_t)op) & 15) == 0)) {
#pragma unroll
      for (int q = 0; q < 4; ++q)
        ((uint4*)op)[q] = make_uint4(v[4 * q], v[4 * q + 1], v[4 * q + 2], v[4 * q + 3]);
    } else {
      for (int b = 0; b < 16; ++b)
        if (j0 + b < a.cols) op[b] = v[b];
    }
  }

  if (a.dig != nullptr) {
    uint32_t planes[4][4];  // [digit t][word q]: digit t of elements 4q .. 4q+3
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const uint32_t w[4] = {digit_word(v[4 * q]), digit_word(v[4 * q + 1]),
                             digit_word(v[4 * q + 2]), digit_word(v[4 * q + 3])};
      uint32_t t4[4];
      digit_transpose4(w, t4);
#pragma unroll
      for (int t = 0; t < 4; ++t) planes[t][q] = t4[t];
    }
    uint4* dp = (uint4*)(a.dig + i * a.pitch + 64 * g);
#pragma unroll
    for (int t = 0; t < 4; ++t) dp[t] = make_uint4(planes[t][0], planes[t][1], planes[t][2], planes[t][3]);
  }
}

// Fast path of the mask pass for rows of a multiple of 4 columns with
// contiguous plaintext: four consecutive lanes share one 16-column digit
// group, lane q owning columns 4q .. 4q+3. A lane reads 4 plaintext values,
// one 16-byte word of u and one Philox block of noise, and forms the four
// digit words of its columns; a transpose across the four lanes (quad
// shuffles) then hands lane q digit plane q of the whole group, so each lane
// stores 16 contiguous bytes and a wave stores 1 KiB contiguous per
// instruction. Every input is read once and every output written once, so
// all accesses are non-temporal (they do not displace cached data).
// XT: 0 none, 1 int8, 2 int32 or ring words. F: which of u, noise, out and
// digits are present (MQ_* bits). Presence is a compile-time choice: with
// run-time tests the loads of x and u were issued one round trip apart.
enum { MQ_U = 1, MQ_NOISE = 2, MQ_OUT = 4, MQ_DIG = 8 };
// Workgroup b covers 1024-column slice b % slices of row b / slices, so
// consecutive workgroups stream consecutive memory (79% of the HBM peak
// measured for the int8 mask pass, against 67% with rows varying fastest).
template <int XT, int F>
__global__ __launch_bounds__(256) void mask_quad_kernel(MaskLaunch a, int64_t lanes_per_row, uint32_t slices) {
  const uint32_t b = blockIdx.x;
  const int64_t i = b / slices;                     // row
  const int64_t l = (int64_t)(b - (uint32_t)i * slices) * 256 + threadIdx.x;   // lane: columns 4 l .. 4 l + 3
  if (l >= lanes_per_row) return;                   // whole quads leave together (lanes_per_row % 4 == 0)
  const int64_t j0 = 4 * l;
  const bool valid = j0 < a.cols;                   // cols % 4 == 0: all four columns valid or all padding
  uint32_t v[4] = {0u, 0u, 0u, 0u};
  if (valid) {
    u32x4 xw = {0u, 0u, 0u, 0u}, uw = {0u, 0u, 0u, 0u};
    if (XT == 1) {
      const uint32_t w = __builtin_nontemporal_load((const uint32_t*)((const int8_t*)a.x + i * a.x_rs + j0));
#pragma unroll
      for (int b = 0; b < 4; ++b) xw[b] = (uint32_t)(int32_t)(int8_t)(w >> (8 * b));
    } else if (XT == 2) {
      xw = __builtin_nontemporal_load((const u32x4*)((const uint32_t*)a.x + i * a.x_rs + j0));
    }
    if (F & MQ_U) uw = __builtin_nontemporal_load((const u32x4*)(a.u + i * a.ldu + j0));
#pragma unroll
    for (int b = 0; b < 4; ++b) v[b] = xw[b] + uw[b];
    if (F & MQ_NOISE) {
      uint32_t e[4];
      sample4_aligned(a.noise, (uint64_t)i * (uint64_t)a.cols + (uint64_t)j0, e);
      v[0] += e[0]; v[1] += e[1]; v[2] += e[2]; v[3] += e[3];
    }
    if (F & MQ_OUT) {
      const u32x4 ov = {v[0], v[1], v[2], v[3]};
      __builtin_nontemporal_store(ov, (u32x4*)(a.out + i * a.ldo + j0));
    }
  }
  if (F & MQ_DIG) {
    uint32_t o[4];
    quad_digit_planes(v, (int)(l & 3), o);
    const u32x4 ov = {o[0], o[1], o[2], o[3]};
    __builtin_nontemporal_store(ov, (u32x4*)(a.dig + i * a.pitch + 16 * l));
  }
}

template <int XT, int F>
void launch_mask_quad(uint32_t slices, const MaskLaunch& a, int64_t lanes_per_row, hipStream_t s) {
  hipLaunchKernelGGL((mask_quad_kernel<XT, F>), dim3((unsigned)(a.rows * slices)), dim3(256), 0, s, a,
                     lanes_per_row, slices);
}

typedef void (*MaskQuadLaunch)(uint32_t, const MaskLaunch&, int64_t, hipStream_t);

template <int XT>
MaskQuadLaunch mask_quad_for(int f) {
  static const MaskQuadLaunch table[16] = {
      launch_mask_quad<XT, 0>,  launch_mask_quad<XT, 1>,  launch_mask_quad<XT, 2>,  launch_mask_quad<XT, 3>,
      launch_mask_quad<XT, 4>,  launch_mask_quad<XT, 5>,  launch_mask_quad<XT, 6>,  launch_mask_quad<XT, 7>,
      launch_mask_quad<XT, 8>,  launch_mask_quad<XT, 9>,  launch_mask_quad<XT, 10>, launch_mask_quad<XT, 11>,
      launch_mask_quad<XT, 12>, launch_mask_quad<XT, 13>, launch_mask_quad<XT, 14>, launch_mask_quad<XT, 15>};
  return table[f & 15];
}

__global__ __launch_bounds__(256) void signs_kernel(RngArgs r, int64_t n, int8_t* out) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t e0 = 4 * i;
  if (e0 >= n) return;
  const uint4 w = philox_block(r, (uint64_t)i);
  const uint32_t ww[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
  for (int q = 0; q < 4; ++q)
    if (e0 + q < n) out[e0 + q] = (ww[q] >> 31) ? (int8_t)-1 : (int8_t)1;
}

// count = 0, ahead of the workgroups that add their partial counts.
__global__ void zero_count_kernel(int64_t* count) { *count = 0; }

// Differing entries of two rows x cols matrices (b null: nonzero entries
// of a): each thread compares
// 4-column groups (grid-stride), a wave and then the workgroup sum their
// counts, and one atomic per workgroup adds the sum to count.
__global__ __launch_bounds__(256) void count_mismatches_kernel(const uint32_t* a, int64_t lda, const uint32_t* b,
                                                               int64_t ldb, int64_t rows, int64_t cols,
                                                               int64_t* count) {
  __shared__ unsigned part[4];
  unsigned n = 0;
  const int64_t per_row = (cols + 3) / 4;
  const int64_t groups = rows * per_row;
  for (int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x; q < groups; q += (int64_t)gridDim.x * 256) {
    const int64_t i = q / per_row;
    const int64_t j = (q - i * per_row) * 4;
    const uint32_t* ar = a + i * lda + j;
    const uint32_t* br = b != nullptr ? b + i * ldb + j : nullptr;
#pragma unroll
    for (int c = 0; c < 4; ++c)
      if (j + c < cols) n += ar[c] != (b != nullptr ? br[c] : 0u) ? 1u : 0u;
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) n += __shfl_xor(n, off);
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = n;
  __syncthreads();
  if (threadIdx.x == 0) {
    const unsigned t = part[0] + part[1] + part[2] + part[3];
    if (t != 0) atomicAdd((unsigned long long*)count, (unsigned long long)t);
  }
}

// y = ym - kc - c elementwise (kc, c optional). c may share memory with y or
// y_f32 element for element: each thread reads its element of c before it
// writes that element.
__global__ __launch_bounds__(256) void unmask_elementwise_kernel(GemmLaunch g) {
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t i = gid / g.N;
  const int64_t j = gid - i * g.N;
  if (i >= g.M) return;
  uint32_t v = g.ym[i * g.ldy + j];
  if (g.kc != nullptr) v -= g.kc[i * g.ldk + j];
  if (g.c != nullptr) v -= g.c[i * g.ldc + j];
  if (g.y != nullptr) g.y[i * g.ldo + j] = (int32_t)v;
  if (g.y_f32 != nullptr) {
    const float f = (float)(int32_t)v * g.s_rows[i] * g.s_cols[j];
    g.y_f32[i * g.ldf + j] = g.bias != nullptr ? __fadd_rn(f, g.bias[j]) : f;
  }
}

}  // namespace

hipError_t launch_mask(const MaskLaunch& a, hipStream_t s) {
  // fast path: see mask_quad_kernel
  const bool x_ok = a.x == nullptr ||
                    (a.x_cs == 1 && a.x_dtype == 0 && a.x_rs % 4 == 0 && ((uintptr_t)a.x & 3) == 0) ||
                    (a.x_cs == 1 && a.x_dtype >= 2 && a.x_rs % 4 == 0 && ((uintptr_t)a.x & 15) == 0);
  const bool u_ok = a.u == nullptr || (a.ldu % 4 == 0 && ((uintptr_t)a.u & 15) == 0);
  const bool o_ok = a.out == nullptr || (a.ldo % 4 == 0 && ((uintptr_t)a.out & 15) == 0);
  const bool n_ok = !a.has_noise || !a.noise.transposed;
  const int64_t lanes_per_row = (a.dig != nullptr) ? 64 * ((a.cols + 63) / 64) / 4 : 4 * ((a.cols + 15) / 16);
  const int64_t blocks_per_row = (lanes_per_row + 255) / 256;
  if (a.cols % 4 == 0 && x_ok && u_ok && o_ok && n_ok && a.rows * blocks_per_row <= 0x7FFFFFFF) {
    if (a.rows == 0 || lanes_per_row == 0) return hipSuccess;
    const uint32_t slices = (uint32_t)blocks_per_row;
    const int f = (a.u != nullptr ? MQ_U : 0) | (a.has_noise ? MQ_NOISE : 0) | (a.out != nullptr ? MQ_OUT : 0) |
                  (a.dig != nullptr ? MQ_DIG : 0);
    if (a.x == nullptr) mask_quad_for<0>(f)(slices, a, lanes_per_row, s);
    else if (a.x_dtype == 0) mask_quad_for<1>(f)(slices, a, lanes_per_row, s);
    else mask_quad_for<2>(f)(slices, a, lanes_per_row, s);
    return hipGetLastError();
  }
  const int64_t groups = (a.dig != nullptr) ? (64 * ((a.cols + 63) / 64)) / 16 : (a.cols + 15) / 16;
  const int64_t threads = a.rows * groups;
  if (threads == 0) return hipSuccess;
  const int64_t blocks = (threads + 255) / 256;
  hipLaunchKernelGGL(mask_kernel, dim3((unsigned)blocks), dim3(256), 0, s, a, groups);
  return hipGetLastError();
}

hipError_t launch_signs(const RngArgs& r, int64_t n, int8_t* out, hipStream_t s) {
  const int64_t threads = (n + 3) / 4;
  if (threads == 0) return hipSuccess;
  hipLaunchKernelGGL(signs_kernel, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, s, r, n, out);
  return hipGetLastError();
}

hipError_t launch_count_mismatches(const uint32_t* a, int64_t lda, const uint32_t* b, int64_t ldb, int64_t rows,
                                   int64_t cols, int64_t* count, hipStream_t s, bool clear_count) {
  if (clear_count) hipLaunchKernelGGL(zero_count_kernel, dim3(1), dim3(1), 0, s, count);
  const int64_t groups = rows * ((cols + 3) / 4);
  if (groups == 0) return hipGetLastError();
  // about 2 groups per thread, at most 1024 workgroups
  int64_t grid = (groups + 511) / 512;
  if (grid > 1024) grid = 1024;
  hipLaunchKernelGGL(count_mismatches_kernel, dim3((unsigned)grid), dim3(256), 0, s, a, lda, b, ldb, rows, cols,
                     count);
  return hipGetLastError();
}

hipError_t launch_unmask_elementwise(const GemmLaunch& g, hipStream_t s) {
  const int64_t threads = g.M * g.N;
  if (threads == 0) return hipSuccess;
  hipLaunchKernelGGL(unmask_elementwise_kernel, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, s, g);
  return hipGetLastError();
}

}  // namespace mosaic
