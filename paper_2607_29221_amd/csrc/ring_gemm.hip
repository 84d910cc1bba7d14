// Ring product over Z_{2^32} on 8-bit MFMA (gfx950).
//
// Both operands arrive as balanced base-256 digits (see mosaic.h). With
// x = sum_i a_i 256^i and y = sum_j b_j 256^j,
//     x y = sum_{i+j<=3} a_i b_j 256^(i+j)   (mod 2^32),
// the ten surviving limb products of the paper's emulation (Section 6.1). The
// kernel groups them by shift s = i + j into four int32 accumulators per
// output (1, 2, 3 and 4 products) and recombines acc_0 + 2^8 acc_1 +
// 2^16 acc_2 + 2^24 acc_3 with wrap-around arithmetic in the epilogue. Each
// digit tile read from LDS feeds up to four MFMAs, so one pass over the
// operands does the work of the paper's ten INT8 GEMM launches.
//
// Accumulator range: a digit product is at most 2^14 in magnitude, so the
// four-product class acc_3 stays below 2^31 for K < 2^15 (checked by the ABI).
//
// Tiling: 256 threads = 4 waves in a 2 x 2 arrangement; block tile 128 x 128,
// wave tile 64 x 64 as 2 x 2 MFMA tiles of 32 x 32 (v_mfma_i32_32x32x32_i8);
// BK = 64 columns per stage, i.e. 256 bytes per row (4 groups x 4 digits x 16
// bytes). Operand tiles are fetched with buffer loads whose descriptor covers
// only the block's valid rows, so rows past M or N read as zero. In LDS each
// row is padded to 272 bytes: 16 lanes reading the same 16-byte chunk of 16
// consecutive rows then touch all 64 banks once, and every fragment address
// is a per-thread base plus an immediate offset. Double-buffered: 136 KiB.
#include "internal.h"

namespace mosaic {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));

constexpr int BM = 128;
constexpr int BN = 128;
constexpr int BKB = 256;             // bytes per row per stage (64 columns x 4 digits)
constexpr int LROW = BKB + 16;       // padded LDS row pitch in bytes
constexpr int NTHREADS = 256;
constexpr int LOADS = BM * (BKB / 16) / NTHREADS;   // 16-byte loads per thread per operand (8)
constexpr int OPB = BM * LROW;       // bytes of one operand stage in LDS
constexpr uint32_t kRsrcWord3 = 0x00020000u;

struct Tile {
  int64_t tm, tn;
};

// Grouped ordering: GROUP_M consecutive row tiles sweep the column tiles
// together, so blocks that run at the same time share operand rows in L2.
__device__ __forceinline__ Tile tile_of(int64_t pid, int64_t tiles_m, int64_t tiles_n) {
  constexpr int64_t GROUP_M = 8;
  const int64_t per_group = GROUP_M * tiles_n;
  const int64_t group = pid / per_group;
  const int64_t first_m = group * GROUP_M;
  const int64_t gm = (tiles_m - first_m) < GROUP_M ? (tiles_m - first_m) : GROUP_M;
  const int64_t in_group = pid - group * per_group;
  Tile t;
  t.tm = first_m + in_group % gm;
  t.tn = in_group / gm;
  return t;
}

__device__ __forceinline__ uint4 lds_read16(const char* lds, int off) {
  return *(const uint4*)(lds + off);
}

template <int EPI>
__global__ __launch_bounds__(NTHREADS, 1) void ring_gemm_kernel(GemmLaunch g) {
  __shared__ __attribute__((aligned(16))) char lds[2 * 2 * OPB];   // [buffer][A/B][row][272 B]

  const int64_t tiles_m = (g.M + BM - 1) / BM;
  const int64_t tiles_n = (g.N + BN - 1) / BN;
  const Tile tile = tile_of(blockIdx.x, tiles_m, tiles_n);
  const int64_t m0 = tile.tm * BM;
  const int64_t n0 = tile.tn * BN;
  const int64_t rows_a = (g.M - m0) < BM ? (g.M - m0) : BM;
  const int64_t rows_b = (g.N - n0) < BN ? (g.N - n0) : BN;

  const __amdgpu_buffer_rsrc_t rsa = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(g.a + m0 * g.a_pitch), (short)0, (int)(rows_a * g.a_pitch), kRsrcWord3);
  const __amdgpu_buffer_rsrc_t rsb = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(g.b + n0 * g.b_pitch), (short)0, (int)(rows_b * g.b_pitch), kRsrcWord3);

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave >> 1;
  const int wn = wave & 1;

  // global -> LDS: thread copies chunk (tid % 16) of rows tid / 16 + 16 p
  const int lchunk = tid & 15;
  const int lrow = tid >> 4;
  const int voff_a = lrow * (int)g.a_pitch + lchunk * 16;
  const int voff_b = lrow * (int)g.b_pitch + lchunk * 16;
  const int step_a = 16 * (int)g.a_pitch;
  const int step_b = 16 * (int)g.b_pitch;
  const int lds_st = lrow * LROW + lchunk * 16;

  // fragment reads: lane reads row (lane % 32) of a 32-row MFMA tile,
  // column group (lane / 32) of the 32-column k-slice
  const int frow = lane & 31;
  const int fgrp = lane >> 5;
  const int lds_fa = (wm * 64 + frow) * LROW + fgrp * 64;
  const int lds_fb = (wn * 64 + frow) * LROW + fgrp * 64;

  v16i acc[2][2][4];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int s = 0; s < 4; ++s)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[i][j][s][v] = 0;

  const int stages = (int)(g.Kp / 64);
  uint4 sa[LOADS], sb[LOADS];

  if (stages > 0) {
#pragma unroll
    for (int p = 0; p < LOADS; ++p) {
      const v4i va = __builtin_bit_cast(v4i, __builtin_amdgcn_raw_buffer_load_b128(rsa, voff_a + p * step_a, 0, 0));
      const v4i vb = __builtin_bit_cast(v4i, __builtin_amdgcn_raw_buffer_load_b128(rsb, voff_b + p * step_b, 0, 0));
      sa[p] = make_uint4(va[0], va[1], va[2], va[3]);
      sb[p] = make_uint4(vb[0], vb[1], vb[2], vb[3]);
    }
#pragma unroll
    for (int p = 0; p < LOADS; ++p) {
      *(uint4*)(lds + lds_st + p * 16 * LROW) = sa[p];
      *(uint4*)(lds + OPB + lds_st + p * 16 * LROW) = sb[p];
    }
  }
  __syncthreads();

  for (int s = 0; s < stages; ++s) {
    const int cur = (s & 1) * 2 * OPB;
    const bool more = (s + 1) < stages;
    if (more) {
      const int kb = (s + 1) * BKB;
#pragma unroll
      for (int p = 0; p < LOADS; ++p) {
        const v4i va = __builtin_bit_cast(v4i, __builtin_amdgcn_raw_buffer_load_b128(rsa, voff_a + p * step_a + kb, 0, 0));
        const v4i vb = __builtin_bit_cast(v4i, __builtin_amdgcn_raw_buffer_load_b128(rsb, voff_b + p * step_b + kb, 0, 0));
        sa[p] = make_uint4(va[0], va[1], va[2], va[3]);
        sb[p] = make_uint4(vb[0], vb[1], vb[2], vb[3]);
      }
    }

#pragma unroll
    for (int h = 0; h < 2; ++h) {          // two 32-column k-slices per stage
      v4i af[2][4], bf[2][4];
#pragma unroll
      for (int i = 0; i < 2; ++i) {
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          const int off = i * 32 * LROW + h * 128 + t * 16;
          const uint4 va = lds_read16(lds + cur, lds_fa + off);
          const uint4 vb = lds_read16(lds + cur + OPB, lds_fb + off);
          af[i][t] = v4i{(int)va.x, (int)va.y, (int)va.z, (int)va.w};
          bf[i][t] = v4i{(int)vb.x, (int)vb.y, (int)vb.z, (int)vb.w};
        }
      }
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
          for (int ta = 0; ta < 4; ++ta)
#pragma unroll
            for (int tb = 0; tb < 4 - ta; ++tb)
              acc[i][j][ta + tb] =
                  __builtin_amdgcn_mfma_i32_32x32x32_i8(af[i][ta], bf[j][tb], acc[i][j][ta + tb], 0, 0, 0);
    }

    if (more) {
      const int nxt = ((s + 1) & 1) * 2 * OPB;
#pragma unroll
      for (int p = 0; p < LOADS; ++p) {
        *(uint4*)(lds + nxt + lds_st + p * 16 * LROW) = sa[p];
        *(uint4*)(lds + nxt + OPB + lds_st + p * 16 * LROW) = sb[p];
      }
    }
    __syncthreads();
  }

  // epilogue: recombine the shift classes and write. Output layout of the
  // 32 x 32 MFMA: register v of lane l holds row 8 (v / 4) + 4 (l / 32) + v % 4,
  // column l % 32.
#pragma unroll
  for (int i = 0; i < 2; ++i) {
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int64_t n = n0 + wn * 64 + j * 32 + (lane & 31);
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int64_t m = m0 + wm * 64 + i * 32 + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
        if (m < g.M && n < g.N) {
          const uint32_t val = (uint32_t)acc[i][j][0][v] + ((uint32_t)acc[i][j][1][v] << 8) +
                               ((uint32_t)acc[i][j][2][v] << 16) + ((uint32_t)acc[i][j][3][v] << 24);
          if (EPI == EPI_STORE) {
            g.c[m * g.ldc + n] = val;
          } else {
            uint32_t y = g.ym[m * g.ldy + n] - val;
            if (g.kc != nullptr) y -= g.kc[m * g.ldk + n];
            if (g.y != nullptr) g.y[m * g.ldo + n] = (int32_t)y;
            if (g.y_f32 != nullptr) g.y_f32[m * g.ldf + n] = (float)(int32_t)y * g.s_rows[m] * g.s_cols[n];
          }
        }
      }
    }
  }
}

}  // namespace

hipError_t launch_ring_gemm(const GemmLaunch& g, EpilogueKind epi, hipStream_t s) {
  const int64_t tiles = ((g.M + BM - 1) / BM) * ((g.N + BN - 1) / BN);
  if (tiles == 0) return hipSuccess;
  if (epi == EPI_STORE)
    hipLaunchKernelGGL(ring_gemm_kernel<EPI_STORE>, dim3((unsigned)tiles), dim3(NTHREADS), 0, s, g);
  else
    hipLaunchKernelGGL(ring_gemm_kernel<EPI_UNMASK>, dim3((unsigned)tiles), dim3(NTHREADS), 0, s, g);
  return hipGetLastError();
}

}  // namespace mosaic
