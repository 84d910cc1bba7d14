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
// Two kernels:
//
// ring_gemm_skinny_kernel (store and accumulate epilogues). The unit of work
// is one (column tile, stage) pair: 128 rows of B (output columns) against
// all rows of A over 64 columns of K. The units are cut into one contiguous
// range per compute unit, so every grid shape keeps the chip busy; a
// workgroup walks its range tile by tile and adds each tile's partial
// product into C with 32-bit atomics (exact in the ring; C is cleared first
// for a plain store). Both operands of a stage are staged in LDS by direct
// buffer-to-LDS loads, three stages resident and loads issued two stages
// ahead, so data in flight costs no registers; the units with a fetch two
// ahead run in a loop with no tests on the unit index and LDS slots taken in
// rotation (one-token products at 4096 x 4096 2-7% faster than with the
// tests and a 64-bit slot modulo in every unit). The waves of a workgroup
// split the tile's columns (32 each, 4 column groups): the A stage is
// fetched once per workgroup and read from LDS by every wave, where a split
// of K between the waves would fetch all of A once per wave and need a
// reduction of the waves' partial products. For A of more than 16 rows a
// second row of 4 waves takes the other half of A's rows (8 waves, two per
// SIMD: one wave's MFMAs run while the other waits at the barrier or on
// LDS), and A of 33-64 rows is padded to 64. Measured against the K-split
// design (B streamed into registers) at the decode and mat-vec shapes:
// 4-10% less time for one token, 20-26% for 16 and 32 tokens, about 50% for
// 64 (35% with one row of waves).
//
// Unmask epilogue. Its output cannot take partial products, so when an
// output buffer of the call (y, else y_f32) shares no memory with any input,
// the product is computed into that buffer by the shared-A kernel and an
// elementwise pass then forms y = ym - kc - product in place (when y is that
// buffer and no fp32 output is asked for, the elementwise pass writes
// y = ym - kc first and the product's partial sums are subtracted from it,
// so y is neither cleared nor read again). Otherwise
// ring_gemm_skinny_ksplit_kernel runs: one workgroup per column tile of 32
// (A of at most 16 rows) or 64 rows of B computes the whole K range, its 4
// waves splitting the stages, streaming their part of B straight into
// registers and summing their partial products in LDS before the epilogue.
// With the short K of unmasking (the rank) that kernel has only N / 32 or
// N / 64 workgroups: at the decode unmask shapes (N 4096 / 14336, rank 1024 /
// 2560) the two-phase path takes 1.5-3.3x less time for 64 tokens, 6-23%
// less for 8, and is within 5% either way for one token; for A of at most
// 16 rows it runs only when the factor is large (see the launcher).
//
// LDS layout (shared-A kernel). A stage row is 256 bytes: 4 groups of 16
// columns, each holding its 4 digit planes in 64 consecutive bytes, i.e. 16
// chunks of 16 bytes. Chunk c of row R sits in slot c ^ (R & 15), so 16
// lanes reading one chunk of 16 consecutive rows touch all 64 banks once. A
// direct load writes 64 consecutive 16-byte slots (4 rows); each lane
// fetches the chunk that belongs to its slot.
//
// Operand fragments. For the 16 x 16 x 64 instruction, lane l supplies row
// l % 16 and sixteen of the 64 k-slots, chosen by h = l / 16. Lane (h, r)
// takes chunk 4 h + t of row r for the fragment of digit t: digit t of
// column group h. A and B use the same k-slot assignment, which is all the
// product needs.
#include "internal.h"

namespace mosaic {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));

constexpr int ROWB = 256;   // bytes per row per stage: 64 columns x 4 digits

// limb pairs (a, b) with a + b <= 3, grouped by the digit of B
__device__ constexpr int kLimbA[10] = {0, 1, 2, 3, 0, 1, 2, 0, 1, 0};
__device__ constexpr int kLimbB[10] = {0, 0, 0, 0, 1, 1, 1, 2, 2, 3};

// ---------------------------------------------------------------------------
// Shared-A kernel (store and accumulate epilogues)

constexpr int SA_WN = 4;                           // waves along the tile's columns
constexpr int SA_NTW = 2;                          // 16-row B tiles per wave
constexpr int SA_BN = SA_WN * SA_NTW * 16;         // B rows per column tile
constexpr int SA_NS = 3;                           // stages resident in LDS

// Direct buffer-to-LDS load of 16 bytes per lane: lane l writes LDS bytes
// [lds_off + 16 l, lds_off + 16 l + 16). Inline assembly, so that the
// compiler, which cannot tell these writes from later LDS reads, does not
// drain every outstanding load before each read; completion is tracked by
// hand (wait_vm) before the barrier that publishes a stage. M0 (the LDS
// base) is set inside the same statement; nothing else in this kernel uses
// M0.
__device__ __forceinline__ void dma16(v4i rs, uint32_t lds_off, int voff, int soff) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, %3 offen lds"
               :: "s"(lds_off), "v"(voff), "s"(rs), "s"(soff) : "memory");
}

// Raw buffer descriptor over [base, base + bytes): out-of-range lanes read 0.
// The arguments are uniform; readfirstlane states it, so the descriptor
// stays in scalar registers as the direct load requires.
__device__ __forceinline__ v4i make_rsrc(const void* base, int64_t bytes) {
  const uint64_t b = (uint64_t)base;
  return v4i{__builtin_amdgcn_readfirstlane((int)(uint32_t)b),
             __builtin_amdgcn_readfirstlane((int)((uint32_t)(b >> 32) & 0xFFFFu)),
             __builtin_amdgcn_readfirstlane((int)bytes), (int)0x00020000u};
}

// s_waitcnt with only the vector-memory counter constrained: vmcnt(N)
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// Workgroup b computes units [units b / grid, units (b + 1) / grid) of the
// tiles x stages (column tile, stage) pairs, tile-major, with WM x 4 waves:
// wave (wm, wn) multiplies A row tiles wm MT / WM .. +MT / WM with B row tiles
// 2 wn, 2 wn + 1 of the column tile. K must be non-zero.
// BW: B arrives as ring words (row pitch b_pitch bytes) instead of digits. A
// stage's 64 words of a row occupy 256 bytes, the size of its digit row, so
// the direct loads and the fragment reads are unchanged: the four 16-byte
// slots a lane reads for a B tile hold the 16 words of one column group,
// and the lane turns them into that group's four digit planes in registers.
// Columns past K read whatever follows in B's rows;
// A's zero digits there cancel them. The stage offset then travels in the
// per-lane offset, which the buffer range check covers, and the range ends
// b_last bytes into B's last row, so that no load leaves the words B holds.
template <int MT, int WM, bool BW = false>
__global__ __launch_bounds__(64 * WM * SA_WN, 1) void ring_gemm_skinny_kernel(GemmLaunch g, int64_t units) {
  constexpr int NW = WM * SA_WN;
  constexpr int MTW = MT / WM;                     // A row tiles per wave
  static_assert(MT % WM == 0, "A row tiles split evenly between the rows of waves");
  constexpr int ASZ = 16 * MT * ROWB;              // A part of a stage
  constexpr int STG = ASZ + SA_BN * ROWB;          // one stage
  static_assert((4 * MT) % NW == 0 && (SA_BN / 4) % NW == 0, "direct loads split evenly between the waves");
  constexpr int QA = 4 * MT / NW;                  // direct loads per wave per stage: A ...
  constexpr int QB = SA_BN / 4 / NW;               // ... and B (1 KiB = 4 rows each)
  constexpr int QU = QA + QB;
  static_assert(SA_NS * STG <= 160 * 1024, "LDS");
  __shared__ __attribute__((aligned(1024))) char lds[SA_NS * STG];

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = wave / SA_WN, wn = wave % SA_WN;
  const int64_t stages = g.Kp / 64;
  const int64_t u0 = units * blockIdx.x / gridDim.x;
  const int64_t cnt = units * (blockIdx.x + 1) / gridDim.x - u0;
  if (cnt <= 0) return;

  // direct loads: wave w fills A rows 4 QA w .. +4 QA and B rows 4 QB w .. +4 QB
  // of every stage
  const int lr = lane >> 4, ls = lane & 15;
  int va[QA], vb[QB];
#pragma unroll
  for (int q = 0; q < QA; ++q) {
    const int R = wave * 4 * QA + 4 * q + lr;
    va[q] = R * (int)g.a_pitch + ((ls ^ (R & 15)) << 4);
  }
#pragma unroll
  for (int q = 0; q < QB; ++q) {
    const int R = wave * 4 * QB + 4 * q + lr;
    vb[q] = R * (int)g.b_pitch + ((ls ^ (R & 15)) << 4);
  }
  const uint32_t lds0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char*)lds;
  const v4i rsa = make_rsrc(g.a, g.M * g.a_pitch);

  // load cursor: (tile, stage) of the next unit to fetch
  int64_t lt = u0 / stages, lst = u0 - lt * stages;
  auto fetch = [&](int slot) {
    const int64_t n0 = lt * SA_BN;
    const int64_t rows_b = (g.N - n0) < SA_BN ? (g.N - n0) : SA_BN;
    const int64_t bbytes = BW ? (rows_b - 1) * g.b_pitch + g.b_last : rows_b * g.b_pitch;
    const v4i rsb = make_rsrc(g.b + n0 * g.b_pitch, bbytes);
    const int soff = (int)lst * ROWB;
    const uint32_t base = lds0 + (uint32_t)slot * STG;
#pragma unroll
    for (int q = 0; q < QA; ++q) dma16(rsa, base + (wave * 4 * QA + 4 * q) * ROWB, va[q], soff);
#pragma unroll
    for (int q = 0; q < QB; ++q) {
      if (BW) dma16(rsb, base + ASZ + (wave * 4 * QB + 4 * q) * ROWB, vb[q] + soff, 0);
      else dma16(rsb, base + ASZ + (wave * 4 * QB + 4 * q) * ROWB, vb[q], soff);
    }
    if (++lst == stages) {
      lst = 0;
      ++lt;
    }
  };

  const int r = lane & 15, h = lane >> 4;
  int fo[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) fo[t] = r * ROWB + (((4 * h + t) ^ r) << 4);

  v4i acc[MTW][SA_NTW][4];
#pragma unroll
  for (int i = 0; i < MTW; ++i)
#pragma unroll
    for (int j = 0; j < SA_NTW; ++j)
#pragma unroll
      for (int c = 0; c < 4; ++c) acc[i][j][c] = v4i{0, 0, 0, 0};

#pragma unroll
  for (int s = 0; s < SA_NS - 1; ++s)
    if (s < cnt) fetch(s);

  int64_t ct = u0 / stages, cst = u0 - ct * stages;   // (tile, stage) being computed
  // one unit: fragments from LDS slot `slot`, the ten limb products, and the
  // tile's partial product added into C after its last stage (or the range's
  // last unit)
  auto unit = [&](int slot, bool last) __attribute__((always_inline)) {
    const char* sa = lds + slot * STG + wm * MTW * 16 * ROWB;
    const char* sb = lds + slot * STG + ASZ + wn * 16 * SA_NTW * ROWB;
    v4i fa[MTW][4], fb[SA_NTW][4];
#pragma unroll
    for (int j = 0; j < SA_NTW; ++j)
#pragma unroll
      for (int t = 0; t < 4; ++t) fb[j][t] = *(const v4i*)(sb + j * 16 * ROWB + fo[t]);
    if (BW) {
      // the four slots a lane reads hold the 16 words of its column group;
      // turn them into the group's four digit planes in registers
#pragma unroll
      for (int j = 0; j < SA_NTW; ++j) {
        uint32_t pl[4][4];
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          const uint32_t v4[4] = {(uint32_t)fb[j][c][0], (uint32_t)fb[j][c][1], (uint32_t)fb[j][c][2],
                                  (uint32_t)fb[j][c][3]};
          uint32_t p4[4];
          digit_planes4(v4, p4);
#pragma unroll
          for (int t = 0; t < 4; ++t) pl[t][c] = p4[t];
        }
#pragma unroll
        for (int t = 0; t < 4; ++t) fb[j][t] = v4i{(int)pl[t][0], (int)pl[t][1], (int)pl[t][2], (int)pl[t][3]};
      }
    }
#pragma unroll
    for (int i = 0; i < MTW; ++i)
#pragma unroll
      for (int t = 0; t < 4; ++t) fa[i][t] = *(const v4i*)(sa + i * 16 * ROWB + fo[t]);

    // consecutive MFMAs share the B fragment and write different accumulators
#pragma unroll
    for (int p = 0; p < 10; ++p)
#pragma unroll
      for (int j = 0; j < SA_NTW; ++j)
#pragma unroll
        for (int i = 0; i < MTW; ++i)
          acc[i][j][kLimbA[p] + kLimbB[p]] = __builtin_amdgcn_mfma_i32_16x16x64_i8(
              fa[i][kLimbA[p]], fb[j][kLimbB[p]], acc[i][j][kLimbA[p] + kLimbB[p]], 0, 0, 0);

    if (++cst == stages || last) {
      // add this tile's partial product into C. Output layout of the 16 x 16
      // MFMA: register v of lane l holds row 4 (l / 16) + v, column l % 16.
      const int64_t n0 = ct * SA_BN + wn * 16 * SA_NTW;
#pragma unroll
      for (int i = 0; i < MTW; ++i)
#pragma unroll
        for (int j = 0; j < SA_NTW; ++j)
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            const uint32_t val = (uint32_t)acc[i][j][0][v] + ((uint32_t)acc[i][j][1][v] << 8) +
                                 ((uint32_t)acc[i][j][2][v] << 16) + ((uint32_t)acc[i][j][3][v] << 24);
            const int64_t m = (wm * MTW + i) * 16 + 4 * h + v;
            const int64_t n = n0 + j * 16 + r;
            if (m < g.M && n < g.N) atomicAdd(&g.c[m * g.ldc + n], g.negate ? 0u - val : val);
#pragma unroll
            for (int c = 0; c < 4; ++c) acc[i][j][c][v] = 0;
          }
      cst = 0;
      ++ct;
    }
  };
  // Unit k has landed once at most the later units this wave already issued
  // are in flight (vector-memory counts return in order; atomics of earlier
  // flushes only make the wait longer). The barrier then publishes
  // everyone's loads of unit k and guarantees that no wave still reads unit
  // k - 1, whose slot the next fetch refills. While the unit SA_NS - 1 ahead
  // exists the loop runs without tests on k; the last units take the
  // general form. Slots rotate 0, 1, .., SA_NS - 1.
  int64_t k = 0;
  int cs = 0;
  for (; k + SA_NS - 1 < cnt; ++k) {
    wait_vm<QU>();
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
    fetch(cs == 0 ? SA_NS - 1 : cs - 1);
    unit(cs, false);
    cs = cs + 1 == SA_NS ? 0 : cs + 1;
  }
  for (; k < cnt; ++k) {
    if (k + 1 < cnt) wait_vm<QU>();
    else wait_vm<0>();
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
    unit(cs, k == cnt - 1);
    cs = cs + 1 == SA_NS ? 0 : cs + 1;
  }
  wait_vm<0>();   // no direct load outlives the workgroup's LDS
}

// ---------------------------------------------------------------------------
// K-split kernel (unmask epilogue)

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

// q[c] holds words 4 c .. 4 c + 3 of a 16-column group  ->  q[t] holds the
// group's digit plane t (byte 4 c + b = digit t of word 4 c + b).
__device__ __forceinline__ void words_to_planes(v4i (&q)[4]) {
  uint32_t pl[4][4];
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    const uint32_t v4[4] = {(uint32_t)q[c][0], (uint32_t)q[c][1], (uint32_t)q[c][2], (uint32_t)q[c][3]};
    uint32_t p4[4];
    digit_planes4(v4, p4);
#pragma unroll
    for (int t = 0; t < 4; ++t) pl[t][c] = p4[t];
  }
#pragma unroll
  for (int t = 0; t < 4; ++t) q[t] = v4i{(int)pl[t][0], (int)pl[t][1], (int)pl[t][2], (int)pl[t][3]};
}

// Workgroup b: column tile b (16 NT rows of B), all stages, split into W
// contiguous parts, one per wave. Load t of a wave reads bytes 64 t .. +64
// of the stage in all 16 rows of a tile (lane (h, r) the 16 bytes at
// 64 t + 16 h of row r), so every load consumes whole 64-byte segments; lane
// group h then holds digit h of column group t in register quad t, and a
// 4 x 4 transpose between lane groups and register quads (two rounds of
// lane-swap instructions) turns that into the fragment of digit t. Each
// wave holds S sets of fragments, so S stages of loads are in flight while
// it multiplies; with more than 16 rows of A the accumulators leave room for
// one set only. Prefetches past the wave's last stage are clamped to that
// stage: the duplicate request hits in cache and the loop needs no branches
// around loads. K must be non-zero.
// AW: A arrives as ring words (a_pitch bytes per row, a_last valid bytes in
// its last row). A stage's 64 words of a row fill the 256 bytes its digits
// would, so lane (h, r) loads the 16 words of column group h (four 16-byte
// loads) and turns them into that group's four digit planes in registers,
// which is the fragment the transpose gives for digits. Words past K within
// a row are whatever follows in memory; B's zero digits there cancel them.
template <int EPI, int MT, int NT, int S, int W, bool AW = false>
__global__ __launch_bounds__(64 * W) void ring_gemm_skinny_ksplit_kernel(GemmLaunch g) {
  constexpr int NOUT = MT * NT * 4;   // output registers per lane
  __shared__ uint32_t red[W][NOUT][64];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int stages = (int)(g.Kp / 64);
  const int64_t n0 = (int64_t)blockIdx.x * (16 * NT);
  const int64_t rows_b = (g.N - n0) < 16 * NT ? (g.N - n0) : 16 * NT;
  const __amdgpu_buffer_rsrc_t rb = rsrc(g.b + n0 * g.b_pitch, rows_b * g.b_pitch);
  const __amdgpu_buffer_rsrc_t ra = rsrc(g.a, AW ? (g.M - 1) * g.a_pitch + g.a_last : g.M * g.a_pitch);

  const int r = lane & 15;
  const int h = lane >> 4;
  int ob[NT], oa[MT];
#pragma unroll
  for (int j = 0; j < NT; ++j) ob[j] = (j * 16 + r) * (int)g.b_pitch + h * 16;
#pragma unroll
  for (int i = 0; i < MT; ++i) oa[i] = (i * 16 + r) * (int)g.a_pitch + (AW ? h * 64 : h * 16);

  // this wave's share [s0, s1) of the stages
  const int per = (stages + W - 1) / W;
  const int s0 = wave * per < stages ? wave * per : stages;
  const int s1 = (s0 + per) < stages ? (s0 + per) : stages;

  v4i acc[MT][NT][4];
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int j = 0; j < NT; ++j)
#pragma unroll
      for (int c = 0; c < 4; ++c) acc[i][j][c] = v4i{0, 0, 0, 0};

  if (s0 < s1) {
    v4i fa[S][MT][4], fb[S][NT][4];

#define KS_LOAD(SET, S)                                                                    \
  do {                                                                                     \
    const int so_ = (S) * ROWB;                                                            \
    _Pragma("unroll") for (int j = 0; j < NT; ++j)                                         \
    _Pragma("unroll") for (int t = 0; t < 4; ++t) fb[SET][j][t] = load16(rb, ob[j] + so_ + 64 * t); \
    _Pragma("unroll") for (int i = 0; i < MT; ++i)                                         \
    _Pragma("unroll") for (int t = 0; t < 4; ++t) fa[SET][i][t] = load16(ra, oa[i] + so_ + (AW ? 16 : 64) * t); \
  } while (0)

#define KS_MFMA(SET)                                                                       \
  do {                                                                                     \
    _Pragma("unroll") for (int j = 0; j < NT; ++j) transpose4(fb[SET][j]);                 \
    _Pragma("unroll") for (int i = 0; i < MT; ++i) {                                       \
      if (AW) words_to_planes(fa[SET][i]);                                                 \
      else transpose4(fa[SET][i]);                                                         \
    }                                                                                      \
    _Pragma("unroll") for (int p = 0; p < 10; ++p)                                         \
    _Pragma("unroll") for (int i = 0; i < MT; ++i)                                         \
    _Pragma("unroll") for (int j = 0; j < NT; ++j)                                         \
      acc[i][j][kLimbA[p] + kLimbB[p]] = __builtin_amdgcn_mfma_i32_16x16x64_i8(            \
          fa[SET][i][kLimbA[p]], fb[SET][j][kLimbB[p]], acc[i][j][kLimbA[p] + kLimbB[p]], 0, 0, 0); \
  } while (0)

    // Position i of the wave's walk visits stage s0 + (i + rot) mod cnt.
    // The rotation differs between neighbouring workgroups, so at any moment
    // they read different parts of A instead of all requesting the same lines
    // (which would queue on a few L2 channels).
    const int cnt = s1 - s0;
    const int rot = (int)(blockIdx.x % (unsigned)cnt);
#define KS_STAGE(i) (s0 + (((i) + rot) < cnt ? ((i) + rot) : ((i) + rot - cnt)))
    if constexpr (S > 1) {
#pragma unroll
      for (int q = 0; q < S; ++q) KS_LOAD(q, KS_STAGE(q < cnt ? q : cnt - 1));
      for (int i = 0; i < cnt; i += S) {
#pragma unroll
        for (int q = 0; q < S; ++q) {
          if (q == 0 || i + q < cnt) KS_MFMA(q);
          KS_LOAD(q, KS_STAGE((i + q + S) < cnt ? (i + q + S) : cnt - 1));
        }
      }
    } else {
      for (int i = 0; i < cnt; ++i) {
        KS_LOAD(0, KS_STAGE(i));
        KS_MFMA(0);
      }
    }
#undef KS_STAGE
#undef KS_LOAD
#undef KS_MFMA
  }

  // recombine the shift classes, then sum the waves' K ranges in LDS
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

  for (int idx = threadIdx.x; idx < NOUT * 64; idx += 64 * W) {
    const int q = idx >> 6, l = idx & 63;
    uint32_t val = 0;
#pragma unroll
    for (int w = 0; w < W; ++w) val += red[w][q][l];
    const int i = q / (NT * 4), j = (q / 4) % NT, v = q % 4;
    const int64_t m = i * 16 + 4 * (l >> 4) + v;
    const int64_t n = n0 + j * 16 + (l & 15);
    if (m < g.M && n < g.N) gemm_epilogue<EPI>(g, m, n, val);
  }
}

// Zeroes the M x N words at c (leading dimension ldc): block (x, y) covers
// columns 1024 x .. 1024 x + 1023 of rows y, y + gridDim.y, ...; each thread
// four consecutive words, one 16-byte store where the row allows it.
__global__ __launch_bounds__(256) void clear_c_kernel(uint32_t* c, int64_t ldc, int64_t M, int64_t N,
                                                      int64_t* zero) {
  if (zero != nullptr && blockIdx.x == 0 && blockIdx.y == 0 && threadIdx.x == 0) *zero = 0;
  const int64_t j = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 4;
  if (j >= N) return;
  for (int64_t row = blockIdx.y; row < M; row += gridDim.y) {
    uint32_t* cr = c + row * ldc + j;
    if (j + 4 <= N && ((uintptr_t)cr & 15) == 0) {
      *(u32x4*)cr = u32x4{0u, 0u, 0u, 0u};
    } else {
      for (int q = 0; q < 4 && j + q < N; ++q) cr[q] = 0u;
    }
  }
}

void launch_clear_c(uint32_t* c, int64_t ldc, int64_t M, int64_t N, hipStream_t s, int64_t* zero = nullptr) {
  if (M <= 0 || N <= 0) return;
  const dim3 grid((unsigned)((N + 1023) / 1024), (unsigned)(M < 65535 ? M : 65535));
  hipLaunchKernelGGL(clear_c_kernel, grid, dim3(256), 0, s, c, ldc, M, N, zero);
}

// Store and accumulate: the (tile, stage) units cut into one range per
// compute unit (at least 2 units each); a plain store clears C first.
template <int MT, int WM, bool BW = false>
hipError_t launch_shared_a(const GemmLaunch& g, EpilogueKind epi, hipStream_t s) {
  const int64_t tiles = (g.N + SA_BN - 1) / SA_BN;
  const int64_t units = tiles * (g.Kp / 64);
  const int64_t cus = compute_units();
  const int64_t grid = cus < (units + 1) / 2 ? cus : (units + 1) / 2;
  if (epi == EPI_STORE) launch_clear_c(g.c, g.ldc, g.M, g.N, s);
  hipLaunchKernelGGL((ring_gemm_skinny_kernel<MT, WM, BW>), dim3((unsigned)grid), dim3(64 * WM * SA_WN), 0, s, g,
                     units);
  return hipGetLastError();
}

// Byte range [lo, hi) touched by a rows x cols matrix (elem bytes per entry,
// leading dimension ld entries); empty for a null pointer.
struct Span {
  uintptr_t lo, hi;
};
Span span(const void* p, int64_t rows, int64_t cols, int64_t ld, int64_t elem) {
  if (p == nullptr || rows <= 0 || cols <= 0) return {0, 0};
  const uintptr_t b = (uintptr_t)p;
  return {b, b + (uintptr_t)(((rows - 1) * ld + cols) * elem)};
}
bool overlap(Span a, Span b) { return a.lo < a.hi && b.lo < b.hi && a.lo < b.hi && b.lo < a.hi; }

// An output of the unmask call that shares no byte with any input (ym, kc,
// the digit factors, the scale and bias vectors) nor with the other output, or null.
uint32_t* unmask_scratch(const GemmLaunch& g, int64_t* ld) {
  const Span in[] = {span(g.ym, g.M, g.N, g.ldy, 4), span(g.kc, g.M, g.N, g.ldk, 4),
                     span(g.a, g.M, 4 * g.Kp, g.a_pitch, 1), span(g.b, g.N, 4 * g.Kp, g.b_pitch, 1),
                     span(g.s_rows, 1, g.M, g.M, 4), span(g.s_cols, 1, g.N, g.N, 4),
                     span(g.bias, 1, g.N, g.N, 4)};
  const Span sy = span(g.y, g.M, g.N, g.ldo, 4), sf = span(g.y_f32, g.M, g.N, g.ldf, 4);
  auto free_of_inputs = [&](Span o) {
    for (const Span& i : in)
      if (overlap(o, i)) return false;
    return true;
  };
  if (g.y != nullptr && free_of_inputs(sy) && !overlap(sy, sf)) {
    *ld = g.ldo;
    return (uint32_t*)g.y;
  }
  if (g.y_f32 != nullptr && free_of_inputs(sf) && !overlap(sf, sy)) {
    *ld = g.ldf;
    return (uint32_t*)g.y_f32;
  }
  return nullptr;
}

template <int EPI, int MT, int NT, int S, int W, bool AW = false>
hipError_t launch_ksplit(const GemmLaunch& g, hipStream_t s) {
  const int64_t tiles = (g.N + 16 * NT - 1) / (16 * NT);
  hipLaunchKernelGGL((ring_gemm_skinny_ksplit_kernel<EPI, MT, NT, S, W, AW>), dim3((unsigned)tiles), dim3(64 * W), 0,
                     s, g);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_ring_gemm_words_b(const GemmLaunch& g, EpilogueKind epi, hipStream_t s) {
  if (g.M <= 0 || g.N <= 0) return hipSuccess;
  if (g.Kp == 0) {
    if (epi == EPI_STORE) launch_clear_c(g.c, g.ldc, g.M, g.N, s);
    return hipGetLastError();
  }
  const int mt = (int)((g.M + 15) / 16);
  if (mt <= 1) return launch_shared_a<1, 1, true>(g, epi, s);
  if (mt == 2) return launch_shared_a<2, 2, true>(g, epi, s);
  return launch_shared_a<4, 2, true>(g, epi, s);
}

hipError_t launch_unmask_words_a(const GemmLaunch& g, hipStream_t s) {
  if (g.M <= 0 || g.N <= 0) return hipSuccess;
  if (g.M > 16) return hipErrorInvalidValue;
  if (g.Kp == 0) return launch_unmask_elementwise(g, s);
  // the single-launch kernel at every factor size: the digit conversion of
  // A it replaces was a launch of its own
  if (g.N <= 16 * compute_units()) return launch_ksplit<EPI_UNMASK, 1, 1, 2, 4, true>(g, s);
  return launch_ksplit<EPI_UNMASK, 1, 2, 2, 4, true>(g, s);
}

hipError_t launch_clear_check(uint32_t* d, int64_t ldd, int64_t rows, int64_t cols, int64_t* count, hipStream_t s) {
  if (rows <= 0 || cols <= 0) {
    hipLaunchKernelGGL(clear_c_kernel, dim3(1), dim3(1), 0, s, d, ldd, int64_t(0), int64_t(0), count);
    return hipGetLastError();
  }
  launch_clear_c(d, ldd, rows, cols, s, count);
  return hipGetLastError();
}

hipError_t launch_ring_gemm_skinny(const GemmLaunch& g, EpilogueKind epi, hipStream_t s) {
  if (g.M <= 0 || g.N <= 0) return hipSuccess;
  const int mt = (int)((g.M + 15) / 16);
  if (g.Kp == 0) {
    // K = 0 leaves only the epilogue: C = 0, C unchanged, or the unmask of a
    // zero product
    if (epi == EPI_UNMASK) return launch_unmask_elementwise(g, s);
    if (epi == EPI_STORE) launch_clear_c(g.c, g.ldc, g.M, g.N, s);
    return hipGetLastError();
  }
  if (epi == EPI_UNMASK) {
    // The two-phase path costs two more launches (clear, elementwise; one,
    // the elementwise pass before the product, when only y is written): for
    // A of at most 16 rows it pays only once the factor read is large (one
    // row against rank-1536 factors of 12-96 MiB, the single launch took
    // 0-20% less device time; at 168 MiB the two were equal).
    const bool two_phase = mt >= 2 || g.N * 4 * g.Kp >= (int64_t(128) << 20);
    int64_t ldp = 0;
    uint32_t* prod = two_phase ? unmask_scratch(g, &ldp) : nullptr;
    if (prod != nullptr) {
      GemmLaunch p = g;
      p.c = prod;
      p.ldc = ldp;
      hipError_t e = hipSuccess;
      if (prod == (uint32_t*)g.y && g.y_f32 == nullptr) {
        // y = ym - kc first, then the product's partial sums subtracted
        // from it atomically: no clear of y and no final pass over it
        GemmLaunch pre = g;
        pre.c = nullptr;
        e = launch_unmask_elementwise(pre, s);
        if (e != hipSuccess) return e;
        p.negate = true;
        if (mt <= 1) return launch_shared_a<1, 1>(p, EPI_ACCUM, s);
        if (mt == 2) return launch_shared_a<2, 2>(p, EPI_ACCUM, s);
        return launch_shared_a<4, 2>(p, EPI_ACCUM, s);
      }
      if (mt <= 1) e = launch_shared_a<1, 1>(p, EPI_STORE, s);
      else if (mt == 2) e = launch_shared_a<2, 2>(p, EPI_STORE, s);
      else e = launch_shared_a<4, 2>(p, EPI_STORE, s);
      if (e != hipSuccess) return e;
      return launch_unmask_elementwise(p, s);
    }
    // NT: 16-row tiles of B per workgroup; S: stages in flight per wave;
    // W: waves splitting K. One tile per workgroup while that leaves no
    // compute unit idle (one row, 2048 x 1536 factor: 7.6 against 10.9 us).
    // For one row, 8 or 16 waves and 3 to 6 stages in flight were slower at
    // every size tried (factors of 12-96 MiB: by 4-50%).
    if (mt <= 1 && g.N <= 16 * compute_units()) return launch_ksplit<EPI_UNMASK, 1, 1, 2, 4>(g, s);
    if (mt <= 1) return launch_ksplit<EPI_UNMASK, 1, 2, 2, 4>(g, s);
    if (mt == 2) return launch_ksplit<EPI_UNMASK, 2, 4, 1, 4>(g, s);
    return launch_ksplit<EPI_UNMASK, 4, 4, 1, 4>(g, s);
  }
  // MT: 16-row tiles of A (33-64 rows padded to 64: faster than 48 rows on
  // one row of waves); WM: rows of 4 waves
  if (mt <= 1) return launch_shared_a<1, 1>(g, epi, s);
  if (mt == 2) return launch_shared_a<2, 2>(g, epi, s);
  return launch_shared_a<4, 2>(g, epi, s);
}

}  // namespace mosaic
