// Ring product C = A B^T over Z_{2^32} for short A (M <= 64 rows): the
// decode-shaped server products of the paper's token-by-token evaluation
// (Section 6), where every byte of the masked weight B is used by only a few
// tokens and the product is bound by streaming B from HBM.
//
// Arithmetic is that of the tiled kernel: balanced base-256 digits, the ten
// limb products with i + j <= 3 grouped by shift class into four int32
// accumulators (the emulation of Section 6.1), recombined with wrap-around
// arithmetic. Here the matrix instruction is v_mfma_i32_16x16x64_i8, so A is
// padded only to 16, 32 or 64 rows.
//
// Work decomposition. The unit of work is one (column tile, stage) pair: 16
// NT rows of B (output columns) against all rows of A over 64 columns of K.
// A workgroup of 4 waves walks a contiguous range of these pairs, one tile
// segment at a time; its waves split each segment's stages into 4
// contiguous parts. Each wave streams its part of B straight from memory
// into registers (no reuse, so no LDS staging), reads the matching part of
// A (shared by all workgroups, so it is served by the caches), and
// multiplies. The partial products of the waves are summed in LDS with
// wrap-around adds, which is exact in the ring. Wide tiles (NT = 2 for A of
// at most 16 rows, 4 above) let each A fragment feed several B fragments:
// every workgroup re-reads all of A, and for 64 tokens those re-reads, not
// B, were the larger share of the traffic. A segment covering a whole tile
// goes through the epilogue; otherwise (the balanced assignment, see
// launch_cfg) partial products are added into C with 32-bit atomics, again
// exact in the ring. Measured against one 16-row tile per workgroup of 8
// waves with whole tiles: 20-24% less time for 8 tokens and 25-40% for 32
// and 64 tokens at the decode shapes.

// Operand fragments. For the 16 x 16 x 64 instruction, lane l supplies row
// l % 16 and sixteen of the 64 k-slots, chosen by l / 16. In the digit layout
// a group of 16 columns keeps its four digit planes in 64 consecutive bytes,
// and a stage (64 columns) of a row is 256 consecutive bytes. Load t of a
// wave reads bytes 64 t .. 64 t + 63 of the stage in all 16 rows (lane l takes
// the 16 bytes at 64 t + 16 (l / 16)), so every load consumes whole 64-byte
// segments; lane group h then holds digit h of column group t in register
// quad t. A 4 x 4 transpose between lane groups and register quads (two
// rounds of lane-swap instructions) turns that into digit t of column group
// h in quad t: the fragment of digit t, with lane group h covering the
// sixteen k-slots of column group h. A and B use the same k-slot assignment,
// which is all the product needs.
//
// Pipelining. For A of up to 16 rows each wave keeps two stages of loads in
// flight (the fragments of the next stage load while the current one
// multiplies); with more rows the accumulators leave no registers for a
// second set of fragments, and the hardware overlaps the waves instead. Prefetches past the
// wave's last stage are clamped to that stage: the duplicate request hits in
// cache and the loop needs no branches around loads.
#include "internal.h"

namespace mosaic {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));

constexpr int NWAVES = 4;
constexpr int NTHREADS = 64 * NWAVES;
constexpr int STAGE_BYTES = 256;   // 64 columns x 4 digits per row

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void* base, int64_t bytes) {
  // out-of-range offsets read as zero
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}

__device__ __forceinline__ v4i load16(__amdgpu_buffer_rsrc_t r, int off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
}

// Swaps dword c of x and y between lane halves (lanes 32..63 of x with lanes
// 0..31 of y), or between 16-lane rows (odd rows of x with even rows of y).
__device__ __forceinline__ void swap32(v4i& x, v4i& y) {
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    const auto r = __builtin_amdgcn_permlane32_swap((unsigned)x[c], (unsigned)y[c], false, false);
    x[c] = (int)r[0];
    y[c] = (int)r[1];
  }
}
__device__ __forceinline__ void swap16(v4i& x, v4i& y) {
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    const auto r = __builtin_amdgcn_permlane16_swap((unsigned)x[c], (unsigned)y[c], false, false);
    x[c] = (int)r[0];
    y[c] = (int)r[1];
  }
}

// q[t] at lane group h  ->  q[h] at lane group t (16-byte blocks).
__device__ __forceinline__ void transpose4(v4i (&q)[4]) {
  swap32(q[0], q[2]);
  swap32(q[1], q[3]);
  swap16(q[0], q[1]);
  swap16(q[2], q[3]);
}

// One segment: the product of all rows of A with B rows n0 .. n0 + 16 NT - 1
// over stages [k0, k1) (64 columns each), written through the epilogue, or
// added into C atomically when `atomic` (EPI_STORE after C was cleared, or
// EPI_ACCUM). Every thread of the workgroup must call it.
template <int MT, int NT, int DB, int EPI>
__device__ __forceinline__ void skinny_segment(const GemmLaunch& g, uint32_t (*red)[MT * NT * 4][64], int64_t n0,
                                               int k0, int k1, bool atomic) {
  constexpr int NOUT = MT * NT * 4;   // output registers per lane
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int64_t rows_b = (g.N - n0) < 16 * NT ? (g.N - n0) : 16 * NT;
  const __amdgpu_buffer_rsrc_t rb = rsrc(g.b + n0 * g.b_pitch, rows_b * g.b_pitch);
  const __amdgpu_buffer_rsrc_t ra = rsrc(g.a, g.M * g.a_pitch);

  const int r = lane & 15;
  const int h = lane >> 4;
  int ob[NT], oa[MT];
#pragma unroll
  for (int j = 0; j < NT; ++j) ob[j] = (j * 16 + r) * (int)g.b_pitch + h * 16;
#pragma unroll
  for (int i = 0; i < MT; ++i) oa[i] = (i * 16 + r) * (int)g.a_pitch + h * 16;

  // this wave's share [s0, s1) of the stages [k0, k1)
  const int per = (k1 - k0 + NWAVES - 1) / NWAVES;
  const int s0 = k0 + wave * per < k1 ? k0 + wave * per : k1;
  const int s1 = (s0 + per) < k1 ? (s0 + per) : k1;

  v4i acc[MT][NT][4];
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int j = 0; j < NT; ++j)
#pragma unroll
      for (int c = 0; c < 4; ++c) acc[i][j][c] = v4i{0, 0, 0, 0};

  if (s0 < s1) {
    v4i fa[1 + DB][MT][4], fb[1 + DB][NT][4];

#define SKINNY_LOAD(SET, S)                                                                \
  do {                                                                                     \
    const int so_ = (S) * STAGE_BYTES;                                                     \
    _Pragma("unroll") for (int j = 0; j < NT; ++j)                                         \
    _Pragma("unroll") for (int t = 0; t < 4; ++t) fb[SET][j][t] = load16(rb, ob[j] + so_ + 64 * t); \
    _Pragma("unroll") for (int i = 0; i < MT; ++i)                                         \
    _Pragma("unroll") for (int t = 0; t < 4; ++t) fa[SET][i][t] = load16(ra, oa[i] + so_ + 64 * t); \
  } while (0)

    // limb pairs (a, b) with a + b <= 3, grouped by the digit of B
#define SKINNY_MFMA(SET)                                                                   \
  do {                                                                                     \
    _Pragma("unroll") for (int j = 0; j < NT; ++j) transpose4(fb[SET][j]);                 \
    _Pragma("unroll") for (int i = 0; i < MT; ++i) transpose4(fa[SET][i]);                 \
    constexpr int ta_[10] = {0, 1, 2, 3, 0, 1, 2, 0, 1, 0};                                \
    constexpr int tb_[10] = {0, 0, 0, 0, 1, 1, 1, 2, 2, 3};                                \
    _Pragma("unroll") for (int p = 0; p < 10; ++p)                                         \
    _Pragma("unroll") for (int i = 0; i < MT; ++i)                                         \
    _Pragma("unroll") for (int j = 0; j < NT; ++j)                                         \
      acc[i][j][ta_[p] + tb_[p]] = __builtin_amdgcn_mfma_i32_16x16x64_i8(                  \
          fa[SET][i][ta_[p]], fb[SET][j][tb_[p]], acc[i][j][ta_[p] + tb_[p]], 0, 0, 0);    \
  } while (0)

    // Position i of the wave's walk visits stage s0 + (i + rot) mod cnt.
    // The rotation differs between neighbouring workgroups, so at any moment
    // they read different parts of A instead of all requesting the same lines
    // (which would queue on a few L2 channels).
    const int cnt = s1 - s0;
    const int rot = (int)(blockIdx.x % (unsigned)cnt);
#define SKINNY_STAGE(i) (s0 + (((i) + rot) < cnt ? ((i) + rot) : ((i) + rot - cnt)))
    if constexpr (DB) {
      SKINNY_LOAD(0, SKINNY_STAGE(0));
      SKINNY_LOAD(DB, SKINNY_STAGE(1 < cnt ? 1 : cnt - 1));
      for (int i = 0; i < cnt; i += 2) {
        SKINNY_MFMA(0);
        SKINNY_LOAD(0, SKINNY_STAGE((i + 2) < cnt ? (i + 2) : cnt - 1));
        if (i + 1 < cnt) SKINNY_MFMA(DB);
        SKINNY_LOAD(DB, SKINNY_STAGE((i + 3) < cnt ? (i + 3) : cnt - 1));
      }
    } else {
      for (int i = 0; i < cnt; ++i) {
        SKINNY_LOAD(0, SKINNY_STAGE(i));
        SKINNY_MFMA(0);
      }
    }
#undef SKINNY_STAGE
#undef SKINNY_LOAD
#undef SKINNY_MFMA
  }

  // recombine the shift classes, then sum the eight K ranges in LDS.
  // Output layout of the 16 x 16 MFMA: register v of lane l holds row
  // 4 (l / 16) + v, column l % 16.
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int j = 0; j < NT; ++j)
#pragma unroll
      for (int v = 0; v < 4; ++v)
        red[wave][(i * NT + j) * 4 + v][lane] =
            (uint32_t)acc[i][j][0][v] + ((uint32_t)acc[i][j][1][v] << 8) +
            ((uint32_t)acc[i][j][2][v] << 16) + ((uint32_t)acc[i][j][3][v] << 24);
  __syncthreads();

  for (int idx = threadIdx.x; idx < NOUT * 64; idx += NTHREADS) {
    const int q = idx >> 6, l = idx & 63;
    uint32_t val = 0;
#pragma unroll
    for (int w = 0; w < NWAVES; ++w) val += red[w][q][l];
    const int i = q / (NT * 4), j = (q / 4) % NT, v = q % 4;
    const int64_t m = i * 16 + 4 * (l >> 4) + v;
    const int64_t n = n0 + j * 16 + (l & 15);
    if (m < g.M && n < g.N) {
      if (atomic) atomicAdd(&g.c[m * g.ldc + n], val);
      else gemm_epilogue<EPI>(g, m, n, val);
    }
  }
}

// Work assignment, one of two; either way a workgroup walks a contiguous
// range [u, u1) of (column tile, stage) pairs, tile by tile, one segment per
// tile it touches:
//  * tiles (units == 0): workgroup b takes column tile b / ks and part b % ks
//    of its K range (ks == 1 for the unmask epilogue, which cannot be split);
//  * balanced (units > 0): the units pairs are cut into gridDim.x equal
//    ranges, so no grid shape leaves a nearly empty last round of
//    workgroups; every segment is added into C atomically.
// K must be non-zero (stages > 0).
template <int MT, int NT, int DB, int EPI, bool BAL>
__global__ __launch_bounds__(NTHREADS) void ring_gemm_skinny_kernel(GemmLaunch g, int ks, int64_t units) {
  __shared__ uint32_t red[NWAVES][MT * NT * 4][64];
  const int64_t stages = g.Kp / 64;
  if constexpr (!BAL) {
    // one segment per workgroup (no loop: the widest tiles use every register)
    const int64_t tile = blockIdx.x / (unsigned)ks;
    const int64_t part = blockIdx.x % (unsigned)ks;
    const int64_t kper = (stages + ks - 1) / ks;
    const int64_t k0 = part * kper < stages ? part * kper : stages;
    const int64_t k1 = (k0 + kper) < stages ? (k0 + kper) : stages;
    skinny_segment<MT, NT, DB, EPI>(g, red, tile * (16 * NT), (int)k0, (int)k1, ks > 1);
    return;
  }
  int64_t u, u1;
  bool atomic;
  if (units == 0) {
    const int64_t tile = blockIdx.x / (unsigned)ks;
    const int64_t part = blockIdx.x % (unsigned)ks;
    const int64_t kper = (stages + ks - 1) / ks;
    const int64_t k0 = part * kper < stages ? part * kper : stages;
    const int64_t k1 = (k0 + kper) < stages ? (k0 + kper) : stages;
    u = tile * stages + k0;
    u1 = tile * stages + k1;
    atomic = ks > 1;
  } else {
    u = units * blockIdx.x / gridDim.x;
    u1 = units * (blockIdx.x + 1) / gridDim.x;
    atomic = true;
  }
  while (u < u1) {
    const int64_t tile = u / stages;
    const int a = (int)(u - tile * stages);
    const int b = (u1 - u) < stages - a ? a + (int)(u1 - u) : (int)stages;
    skinny_segment<MT, NT, DB, EPI>(g, red, tile * (16 * NT), a, b, atomic);
    u += b - a;
    __syncthreads();   // the next segment reuses red
  }
}

__global__ __launch_bounds__(256) void clear_c_kernel(uint32_t* c, int64_t ldc, int64_t M, int64_t N) {
  const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (e < M * N) c[(e / N) * ldc + e % N] = 0u;
}


// Work assignment per launch. The unmask epilogue runs column tiles whole
// (its partial products cannot be added into the output). The store and
// accumulate epilogues use the balanced assignment over one workgroup per
// compute unit (each with at least 4 stages), except that for A of at most
// 16 rows with between 5/8 of and as many column tiles as compute units
// whole tiles are faster (a sweep over the decode and mat-vec shapes: the
// balanced assignment gained 10-35% where tiles exceed the compute units or
// A has 32 or 64 rows, and lost 5-15% with 176-208 tiles; more workgroups
// per compute unit were slower; with 64 tiles whole tiles left three
// quarters of the compute units idle, 2.5x slower). A plain store with partial products added
// atomically clears C first. K = 0 leaves only the epilogue: C = 0, C
// unchanged, or the unmask of a zero product.
template <int MT, int NT, int DB, int EPI>
hipError_t launch_cfg(const GemmLaunch& g, hipStream_t s) {
  const int64_t tiles = (g.N + 16 * NT - 1) / (16 * NT);
  const int64_t stages = g.Kp / 64;
  const dim3 block(NTHREADS);
  if (stages == 0) {
    if (EPI == EPI_UNMASK) return launch_unmask_elementwise(g, s);
    if (EPI == EPI_STORE)
      hipLaunchKernelGGL(clear_c_kernel, dim3((unsigned)((g.M * g.N + 255) / 256)), dim3(256), 0, s, g.c, g.ldc,
                         g.M, g.N);
    return hipGetLastError();
  }
  const int64_t cus = compute_units();
  const int64_t units = tiles * stages;
  if (EPI == EPI_UNMASK || (MT == 1 && tiles <= cus && 8 * tiles >= 5 * cus) || units < 8) {
    hipLaunchKernelGGL((ring_gemm_skinny_kernel<MT, NT, DB, EPI, false>), dim3((unsigned)tiles), block, 0, s, g, 1,
                       (int64_t)0);
    return hipGetLastError();
  }
  const int64_t grid = cus < units / 4 ? cus : units / 4;
  if (EPI == EPI_STORE)
    hipLaunchKernelGGL(clear_c_kernel, dim3((unsigned)((g.M * g.N + 255) / 256)), dim3(256), 0, s, g.c, g.ldc, g.M,
                       g.N);
  hipLaunchKernelGGL((ring_gemm_skinny_kernel<MT, NT, DB, EPI, true>), dim3((unsigned)grid), block, 0, s, g, 1,
                     units);
  return hipGetLastError();
}

template <int EPI>
hipError_t launch_epi(const GemmLaunch& g, hipStream_t s) {
  // MT: 16-row tiles of A (A padded to 16, 32 or 64 rows); NT: 16-row tiles
  // of B per workgroup; DB: double-buffered fragments.
  const int mt = (int)((g.M + 15) / 16);
  if (mt <= 1) return launch_cfg<1, 2, 1, EPI>(g, s);
  if (mt == 2) return launch_cfg<2, 4, 0, EPI>(g, s);
  return launch_cfg<4, 4, 0, EPI>(g, s);
}

}  // namespace

hipError_t launch_ring_gemm_skinny(const GemmLaunch& g, EpilogueKind epi, hipStream_t s) {
  if (g.M <= 0 || g.N <= 0) return hipSuccess;
  if (epi == EPI_STORE) return launch_epi<EPI_STORE>(g, s);
  if (epi == EPI_ACCUM) return launch_epi<EPI_ACCUM>(g, s);
  return launch_epi<EPI_UNMASK>(g, s);
}

}  // namespace mosaic
