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
// four-product class acc_3 stays below 2^31 for K < 2^15; the ABI splits
// longer inner dimensions into chunks whose products are added into C
// (EPI_ACCUM).
//
// Work decomposition. A block of 512 threads (8 waves, two per SIMD) owns a
// 128 x 128 output tile; wave w computes rows 64 (w / 4) .. +64 and columns
// 32 (w % 4) .. +32 as two 32 x 32 tiles of v_mfma_i32_32x32x32_i8, holding
// 2 tiles x 4 shift classes x 16 = 128 accumulator registers. Two waves per
// SIMD let one wave's MFMAs run while the other waits at a barrier or on LDS.
//
// Pipeline. The K dimension is consumed in stages of 32 columns (128 bytes
// per row per operand). Four stages live in LDS at once (4 x 32 KiB) and are
// filled by direct buffer-to-LDS loads issued four stages ahead: stage s's
// fragments are read into registers during stage s-1, so once the barrier
// before stage s has passed, its slot is free and the loads of stage s+4 go
// there. Each wave runs a stage as four groups of 5 MFMAs, pinned by
// scheduling barriers: the 12 LDS reads of stage s+1's fragments follow the
// first three groups (four each), so they have completed by the time the
// next barrier needs them, and one of the wave's 4 direct loads follows
// each group (whole bench steps over the three server shapes 1.2-1.6%
// faster than with the 4 loads after the first two groups, 0.3-0.5% faster
// than with one load and three reads after every group, 4% faster than with
// six reads after each of the first two). The fragments are double-buffered in
// registers. One barrier per stage publishes stage s+1 and retires the slot
// of stage s, which the loads of stage s then refill. All stages but the
// last four run in a loop with no tests (every stage refills and reads),
// four stages per iteration. LDS holds the A tiles of the four slots first
// and then their B tiles (16 KiB each), so that every fragment read
// addresses its slot and tile by an immediate offset from one of the
// lane's eight fragment offsets: that loop computes no addresses in vector
// registers (0.8% faster whole bench steps than slots of A and B together,
// whose third and fourth slots lie beyond the 64 KiB offset range).
//
// LDS rows are 128 bytes (8 chunks of 16 bytes); chunk c of row R sits in
// slot c ^ ((R >> 1) & 7). Sixteen lanes reading one chunk of 16 consecutive
// rows then cover all 64 banks once. A direct load writes 64 consecutive
// 16-byte slots (8 rows), so each lane fetches the chunk that belongs to its
// slot. Operand tiles are addressed through buffer descriptors that cover only
// the block's valid rows: rows past M or N read as zero and never fault.
//
// Epilogue. The recombined tile is staged in the (then idle) LDS and written
// in 16-byte chunks along rows (gemm_tile_epilogue): EPI_STORE writes C,
// EPI_ACCUM adds to C, EPI_UNMASK forms Y = Y' - K_c - C and optionally the
// dequantised fp32 result.
#include "internal.h"

namespace mosaic {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));

constexpr int BM = 128;              // block tile rows (A)
constexpr int BN = 128;              // block tile rows (B) = output columns
constexpr int NTHREADS = 512;
constexpr int BK = 32;               // columns per stage
constexpr int ROWB = BK * 4;         // bytes per row per stage
constexpr int OPS = BM * ROWB;       // one operand stage in LDS (16 KiB)
constexpr int STAGE = 2 * OPS;       // A and B (32 KiB)
constexpr int NSTAGE = 4;            // stages resident in LDS
constexpr uint32_t kRsrcWord3 = 0x00020000u;

struct Tile {
  int64_t tm, tn;
};

// Tile order. Workgroups are dispatched to the 8 XCDs round-robin by id, and
// each XCD has its own L2. The id is first remapped so that XCD x owns a
// contiguous chunk of the logical order (ids x, x+8, x+16, ... become
// consecutive), then the logical order is grouped: GROUP_M row tiles sweep
// the column tiles together. The blocks an XCD runs at once thus cover a
// compact patch of the output, whose operand slices are shared in that XCD's
// L2; XCDs that own the same columns for different row groups sweep them at
// the same pace, so B is shared in the last-level cache as well. Both maps
// are bijections of [0, tiles); correctness does not depend on dispatch
// order.
__device__ __forceinline__ int64_t xcd_order(int64_t pid, int64_t tiles) {
  constexpr int64_t NXCD = 8;
  const int64_t xcd = pid % NXCD;
  const int64_t local = pid / NXCD;
  const int64_t q = tiles / NXCD, r = tiles % NXCD;
  return xcd * q + (xcd < r ? xcd : r) + local;
}

__device__ __forceinline__ Tile tile_at(int64_t lin, int64_t tiles_m, int64_t tiles_n) {
  constexpr int64_t GROUP_M = 8;
  const int64_t per_group = GROUP_M * tiles_n;
  const int64_t group = lin / per_group;
  const int64_t first_m = group * GROUP_M;
  const int64_t gm = (tiles_m - first_m) < GROUP_M ? (tiles_m - first_m) : GROUP_M;
  const int64_t in_group = lin - group * per_group;
  Tile t;
  t.tm = first_m + in_group % gm;
  t.tn = in_group / gm;
  return t;
}

// Direct buffer-to-LDS load of 16 bytes per lane: lane l of the wave writes
// LDS bytes [lds_off + 16 l, lds_off + 16 l + 16). Issued as inline assembly
// so that the compiler, which cannot tell these writes from later LDS reads,
// does not drain every outstanding load before each read; completion is
// tracked by hand with s_waitcnt vmcnt before the barrier that publishes a
// stage. M0 (the LDS base) is set inside the same statement; nothing else in
// this kernel uses M0.
__device__ __forceinline__ void dma16(v4i rs, uint32_t lds_off, int voff, int soff) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, %3 offen lds"
               :: "s"(lds_off), "v"(voff), "s"(rs), "s"(soff) : "memory");
}

// Raw buffer descriptor over [base, base + bytes): out-of-range lanes read 0.
__device__ __forceinline__ v4i make_rsrc(const void* base, int64_t bytes) {
  const uint64_t b = (uint64_t)base;
  return v4i{(int)(uint32_t)b, (int)((uint32_t)(b >> 32) & 0xFFFFu), (int)bytes, (int)kRsrcWord3};
}

// s_waitcnt with only the vector-memory counter constrained: at most 4 n
// direct loads of this wave (n stages) may still be in flight.
__device__ __forceinline__ void wait_loads(int n) {
  if (n >= 3) __builtin_amdgcn_s_waitcnt(0x0F7C);        // vmcnt(12)
  else if (n == 2) __builtin_amdgcn_s_waitcnt(0x0F78);   // vmcnt(8)
  else if (n == 1) __builtin_amdgcn_s_waitcnt(0x0F74);   // vmcnt(4)
  else __builtin_amdgcn_s_waitcnt(0x0F70);               // vmcnt(0)
}

__device__ __forceinline__ int imin(int a, int b) { return a < b ? a : b; }

// Adds a TM x TN tile held in LDS (row pitch TROW words) into C with 32-bit
// atomics (wrap-around adds: exact over the ring), chunks of 4 columns as in
// gemm_tile_epilogue.
template <int TM, int TN, int NT, int TROW>
__device__ __forceinline__ void gemm_tile_atomic_add(const GemmLaunch& g, const uint32_t* tile, int64_t m0,
                                                     int64_t n0, int tid) {
  constexpr int CPR = TN / 4;
  constexpr int PER = TM * CPR / NT;
#pragma unroll
  for (int k = 0; k < PER; ++k) {
    const int c = tid + NT * k;
    const int r = c / CPR;
    const int64_t m = m0 + r;
    const int64_t n = n0 + 4 * (c % CPR);
    if (m >= g.M || n >= g.N) continue;
    const uint4 a = *(const uint4*)(tile + r * TROW + 4 * (c % CPR));
    uint32_t* cr = g.c + m * g.ldc + n;
    atomicAdd(cr, a.x);
    if (n + 1 < g.N) atomicAdd(cr + 1, a.y);
    if (n + 2 < g.N) atomicAdd(cr + 2, a.z);
    if (n + 3 < g.N) atomicAdd(cr + 3, a.w);
  }
}

// Workgroup b < tiles - split_tiles computes a whole tile, in the XCD-aware
// order over those tiles. The last split_tiles tiles of the logical order
// run as split_k pieces each (workgroup full + p: piece p / split_tiles of
// tile full + p % split_tiles), each piece a contiguous range of stage
// pairs, added into C atomically; C is cleared for those tiles first when the
// result is stored (launch_ring_gemm).
// SPLIT: compiled in only for launches with split tiles, so that the
// whole-tile kernel keeps a compile-time stage origin of 0.
template <int EPI, int VEC, bool SPLIT>
__global__ __launch_bounds__(NTHREADS, 1) void ring_gemm_kernel(GemmLaunch g) {
  __shared__ __attribute__((aligned(1024))) char lds[NSTAGE * STAGE];

  const int64_t tiles_m = (g.M + BM - 1) / BM;
  const int64_t tiles_n = (g.N + BN - 1) / BN;
  const int64_t full = SPLIT ? tiles_m * tiles_n - g.split_tiles : tiles_m * tiles_n;
  const int total = (int)(g.Kp / BK);   // even: Kp is a multiple of 64
  const bool piece = SPLIT && (int64_t)blockIdx.x >= full;
  const int64_t p = (int64_t)blockIdx.x - full;
  const int64_t q = piece ? p / g.split_tiles : 0;
  const int64_t lin = piece ? full + (p - q * g.split_tiles) : xcd_order(blockIdx.x, full);
  const int s0 = piece ? 2 * (int)((int64_t)(total / 2) * q / g.split_k) : 0;
  const int stages = piece ? 2 * (int)((int64_t)(total / 2) * (q + 1) / g.split_k) - s0 : total;
  const Tile tile = tile_at(lin, tiles_m, tiles_n);
  const int64_t m0 = tile.tm * BM;
  const int64_t n0 = tile.tn * BN;
  const int64_t rows_a = (g.M - m0) < BM ? (g.M - m0) : BM;
  const int64_t rows_b = (g.N - n0) < BN ? (g.N - n0) : BN;
  // a piece's operands start at its first stage; the ranges end where the
  // tile's rows end
  const v4i rsa = make_rsrc(g.a + m0 * g.a_pitch + s0 * ROWB, rows_a * g.a_pitch - s0 * ROWB);
  const v4i rsb = make_rsrc(g.b + n0 * g.b_pitch + s0 * ROWB, rows_b * g.b_pitch - s0 * ROWB);

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 2;
  const int wn = wave & 3;

  // direct loads: wave w fills rows 16 w + 8 q .. +8 (q = 0, 1) of A and of B
  int voff[4];   // A q0, B q0, A q1, B q1
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const int R = wave * 16 + q * 8 + (lane >> 3);
    const int c = (lane & 7) ^ ((R >> 1) & 7);
    voff[2 * q] = R * (int)g.a_pitch + c * 16;
    voff[2 * q + 1] = R * (int)g.b_pitch + c * 16;
  }
  const uint32_t lds_wave =
      (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char*)lds + wave * 16 * ROWB;

  // fragment reads: lane reads row (lane % 32) of a 32-row tile, chunk
  // 4 (lane / 32) + t for digit t
  const int rr = lane & 31;
  const int f = (rr >> 1) & 7;
  int fo[8];     // A digits 0..3, B digits 0..3
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const int p = ((lane >> 5) * 4 + t) ^ f;
    fo[t] = (wm * 64 + rr) * ROWB + p * 16;
    fo[4 + t] = NSTAGE * OPS + (wn * 32 + rr) * ROWB + p * 16;
  }

  v16i acc[2][4];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int s = 0; s < 4; ++s)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][s][v] = 0;

  v4i fa[2][2][4], fb[2][4];             // [register set][tile][digit], [register set][digit]

#define MOSAIC_DMA(S, k)                                                                   \
  dma16(((k) & 1) ? rsb : rsa,                                                            \
        lds_wave + ((S) & (NSTAGE - 1)) * OPS + ((k) & 1) * NSTAGE * OPS + ((k) >> 1) * 8 * ROWB, voff[k], \
        (S) * ROWB)

#define MOSAIC_READ(S, SET, idx)                                                           \
  do {                                                                                     \
    const char* base_ = lds + ((S) & (NSTAGE - 1)) * OPS;                                  \
    if ((idx) < 8) {                                                                       \
      const int i_ = (idx) >> 2, t_ = (idx) & 3;                                           \
      const uint4 v_ = *(const uint4*)(base_ + i_ * 32 * ROWB + fo[t_]);                   \
      fa[SET][i_][t_] = v4i{(int)v_.x, (int)v_.y, (int)v_.z, (int)v_.w};                   \
    } else {                                                                               \
      const int t_ = (idx) - 8;                                                            \
      const uint4 v_ = *(const uint4*)(base_ + fo[4 + t_]);                                \
      fb[SET][t_] = v4i{(int)v_.x, (int)v_.y, (int)v_.z, (int)v_.w};                       \
    }                                                                                      \
  } while (0)

  // Keeps fragments in VGPRs (the accumulators own the AGPRs) and makes the
  // wave wait for its outstanding LDS reads of that set.
#define MOSAIC_PIN(SET)                                                                    \
  do {                                                                                     \
    _Pragma("unroll") for (int i = 0; i < 2; ++i)                                          \
    _Pragma("unroll") for (int t = 0; t < 4; ++t) asm volatile("" : "+v"(fa[SET][i][t]));  \
    _Pragma("unroll") for (int t = 0; t < 4; ++t) asm volatile("" : "+v"(fb[SET][t]));     \
  } while (0)

  // MFMA n (0..19) of a stage: tile n % 2, limb pair n / 2. The pairs run
  // grouped by the digit of B (b_0 with a_0..a_3, then b_1, b_2, b_3), so
  // consecutive MFMAs share the B fragment in runs of 8, 6, 4 and 2; the
  // matrix cores draw less power when an operand does not change, which on
  // uniform digits gave 1-7% more throughput than orders that switch both
  // operands. The two tiles alternate, so no MFMA reads the accumulator
  // written by the one just before it.
#define MOSAIC_MFMA(SET, n)                                                                \
  do {                                                                                     \
    constexpr int ta_[10] = {0, 1, 2, 3, 0, 1, 2, 0, 1, 0};                                \
    constexpr int tb_[10] = {0, 0, 0, 0, 1, 1, 1, 2, 2, 3};                                \
    const int i_ = (n) % 2, a_ = ta_[(n) / 2], b_ = tb_[(n) / 2];                          \
    acc[i_][a_ + b_] =                                                                     \
        __builtin_amdgcn_mfma_i32_32x32x32_i8(fa[SET][i_][a_], fb[SET][b_], acc[i_][a_ + b_], 0, 0, 0); \
  } while (0)

  // group g of a stage: MFMAs 5g .. 5g+4, then direct load g of stage S+4
  // and (g < 3) fragment reads 4g .. 4g+3 of stage S+1
#define MOSAIC_STAGE(CUR, NXT, S) MOSAIC_STAGE_IF(CUR, NXT, S, (S) + NSTAGE < stages, (S) + 1 < stages)
#define MOSAIC_STAGE_IF(CUR, NXT, S, REFILL, NEXT)                                         \
  do {                                                                                     \
    const bool refill_ = (REFILL);                                                         \
    const bool next_ = (NEXT);                                                             \
    _Pragma("unroll") for (int gq = 0; gq < 4; ++gq) {                                     \
      _Pragma("unroll") for (int u = 0; u < 5; ++u) MOSAIC_MFMA(CUR, gq * 5 + u);          \
      if (refill_) {                                                                       \
        MOSAIC_DMA((S) + NSTAGE, gq);                                                      \
      }                                                                                    \
      if (gq < 3 && next_) {                                                               \
        _Pragma("unroll") for (int r = 0; r < 4; ++r) MOSAIC_READ((S) + 1, NXT, 4 * gq + r); \
      }                                                                                    \
      __builtin_amdgcn_sched_barrier(0);                                                   \
    }                                                                                      \
  } while (0)

  // prologue: stages 0..3 in flight, stage 0 published and read
  for (int s = 0; s < NSTAGE; ++s)
    if (s < stages) {
#pragma unroll
      for (int k = 0; k < 4; ++k) MOSAIC_DMA(s, k);
    }
  if (stages > 0) {
    wait_loads(imin(NSTAGE - 1, stages - 1));
    __builtin_amdgcn_s_barrier();
#pragma unroll
    for (int k = 0; k < 12; ++k) MOSAIC_READ(0, 0, k);
  }

  // Before stage S: this wave's loads of stage S+1 have landed (loads of up
  // to stage S+3 issued, at most two later stages in flight) and its reads of
  // stage S have completed (the pin); the barrier then makes stage S+1
  // visible to every wave and guarantees nobody still reads stage S's slot,
  // which stage S's loads refill with stage S+4.
  // The steady state, where every stage refills its slot and reads the next
  // one, runs as a loop without conditions: one basic block per four stages
  // (slots 0..3 in turn), which the scheduler interleaves freely within the
  // pinned groups (the server products 1.5-3% faster than with the tests
  // inside every stage). The last four stages of a multiple of four run as
  // straight-line code with their waits fixed (bench steps 0.4-0.6% faster
  // than through the general loop, mostly from the short Init X and unmask
  // products); other remainders, and stage counts below eight, take the
  // general loop.
  int it = 0;
  for (; NSTAGE * it + 2 * NSTAGE <= stages; ++it) {
    const int s4 = NSTAGE * it;
#pragma unroll
    for (int h = 0; h < NSTAGE; h += 2) {
      wait_loads(NSTAGE - 2);
      MOSAIC_PIN(0);
      __builtin_amdgcn_s_barrier();
      MOSAIC_STAGE_IF(0, 1, s4 + h, true, true);
      wait_loads(NSTAGE - 2);
      MOSAIC_PIN(1);
      __builtin_amdgcn_s_barrier();
      MOSAIC_STAGE_IF(1, 0, s4 + h + 1, true, true);
    }
  }
  int s = NSTAGE * it;
  if (it > 0 && stages - s == NSTAGE) {
    // the last four stages when the stage count is a multiple of four: no
    // refills, the waits shrink as the loads in flight run out
    wait_loads(2);
    MOSAIC_PIN(0);
    __builtin_amdgcn_s_barrier();
    MOSAIC_STAGE_IF(0, 1, s, false, true);
    wait_loads(1);
    MOSAIC_PIN(1);
    __builtin_amdgcn_s_barrier();
    MOSAIC_STAGE_IF(1, 0, s + 1, false, true);
    wait_loads(0);
    MOSAIC_PIN(0);
    __builtin_amdgcn_s_barrier();
    MOSAIC_STAGE_IF(0, 1, s + 2, false, true);
    MOSAIC_PIN(1);
    MOSAIC_STAGE_IF(1, 0, s + 3, false, false);
    s = stages;
  }
  for (; s < stages; s += 2) {
    wait_loads(imin(NSTAGE - 2, stages - 2 - s));
    MOSAIC_PIN(0);
    __builtin_amdgcn_s_barrier();
    MOSAIC_STAGE(0, 1, s);
    if (s + 2 < stages) wait_loads(imin(NSTAGE - 2, stages - 3 - s));
    MOSAIC_PIN(1);
    if (s + 2 < stages) __builtin_amdgcn_s_barrier();
    MOSAIC_STAGE(1, 0, s + 1);
  }
  __builtin_amdgcn_s_waitcnt(0x0F70);   // no direct load outlives the loop
#undef MOSAIC_DMA
#undef MOSAIC_READ
#undef MOSAIC_PIN
#undef MOSAIC_MFMA
#undef MOSAIC_STAGE
#undef MOSAIC_STAGE_IF

  // epilogue: recombine the shift classes and write. Output layout of the
  // 32 x 32 MFMA: register v of lane l holds row 8 (v / 4) + 4 (l / 32) + v % 4,
  // column l % 32.
  // Recombine the shift classes and stage the 128 x 128 tile in LDS (rows
  // padded to 132 words so the two rows a wave writes per instruction fall in
  // different banks), then write it out in 16-byte chunks along rows: thread
  // t takes chunks t + 512 k (row c / 32, columns 4 (c % 32) .. + 3), so each
  // wave instruction covers two whole 512-byte tile rows. All loads of the
  // unmask epilogue (Y', K_c, scales) are issued before its first store.
  __builtin_amdgcn_s_barrier();                 // every wave is done reading stage data
  uint32_t* ctile = (uint32_t*)lds;
  constexpr int TROW = BN + 4;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int r = wm * 64 + i * 32 + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
      const int c = wn * 32 + (lane & 31);
      ctile[r * TROW + c] = (uint32_t)acc[i][0][v] + ((uint32_t)acc[i][1][v] << 8) +
                           ((uint32_t)acc[i][2][v] << 16) + ((uint32_t)acc[i][3][v] << 24);
    }
  }
  __syncthreads();
  if (EPI != EPI_UNMASK && piece) gemm_tile_atomic_add<BM, BN, NTHREADS, TROW>(g, ctile, m0, n0, tid);
  else gemm_tile_epilogue<EPI, VEC, BM, BN, NTHREADS, TROW>(g, ctile, m0, n0, tid);
}

// C = 0 over the last split_tiles tiles of the logical order (one workgroup
// per tile).
__global__ __launch_bounds__(256) void clear_split_tiles_kernel(GemmLaunch g) {
  const int64_t tiles_m = (g.M + BM - 1) / BM;
  const int64_t tiles_n = (g.N + BN - 1) / BN;
  const Tile tile = tile_at(tiles_m * tiles_n - g.split_tiles + blockIdx.x, tiles_m, tiles_n);
  const int64_t m0 = tile.tm * BM, n0 = tile.tn * BN;
  for (int e = threadIdx.x; e < BM * BN; e += 256) {
    const int64_t m = m0 + e / BN, n = n0 + e % BN;
    if (m < g.M && n < g.N) g.c[m * g.ldc + n] = 0u;
  }
}

// Tiles to split and pieces per tile for a launch of `tiles` whole tiles
// over `cus` compute units. Only the last, partial round of tiles is split,
// and only when it would leave at least half of the compute units idle: the
// chip is power-limited on uniform digits, so a last round on three quarters
// of the units runs at higher clocks, and splitting it measured no faster
// (2048 x 9728 x 8192: 1.22 ms whole, 1.24-1.26 ms with the last 192 tiles in
// four pieces). With a round costing one tile's stages plus a fixed cost per
// workgroup (its prologue and epilogue, taken as 6 stages) and the clear
// before a store (5 stages), split_k pieces of the tail's tiles take
// ceil(tail split_k / cus) rounds of stages / split_k + 6; pieces keep at
// least two stage pairs.
void choose_split(int64_t tiles, int64_t stages, int64_t cus, bool store, int64_t* split_tiles, int* split_k) {
  *split_tiles = 0;
  *split_k = 1;
  if (cus <= 0) return;
  const int64_t tail = tiles % cus;
  if (tail == 0 || 2 * tail >= cus) return;
  constexpr int64_t kFixed = 6, kClear = 5;
  int64_t best = stages + kFixed;
  for (int k : {2, 3, 4, 6, 8}) {
    if (stages / 2 < 2 * (int64_t)k) break;
    const int64_t rounds = (tail * k + cus - 1) / cus;
    const int64_t cost = rounds * (stages / k + kFixed) + (store ? kClear : 0);
    if (cost < best) {
      best = cost;
      *split_k = k;
    }
  }
  if (*split_k > 1) *split_tiles = tail;
}

}  // namespace

hipError_t launch_ring_gemm(const GemmLaunch& g, EpilogueKind epi, hipStream_t s) {
  if (g.M <= SKINNY_MAX_M) return launch_ring_gemm_skinny(g, epi, s);
  const int64_t tiles = ((g.M + BM - 1) / BM) * ((g.N + BN - 1) / BN);
  if (tiles == 0) return hipSuccess;
  GemmLaunch gs = g;
  gs.split_tiles = 0;
  gs.split_k = 1;
  if (epi != EPI_UNMASK)   // the unmask epilogue needs the whole product of a tile
    choose_split(tiles, g.Kp / BK, compute_units(), epi == EPI_STORE, &gs.split_tiles, &gs.split_k);
  if (gs.split_tiles > 0 && epi == EPI_STORE)
    hipLaunchKernelGGL(clear_split_tiles_kernel, dim3((unsigned)gs.split_tiles), dim3(256), 0, s, gs);
  const dim3 grid((unsigned)(tiles + gs.split_tiles * (gs.split_k - 1)));
  const bool vec = gemm_epilogue_vectorizable(g, epi);
  const bool split = gs.split_tiles > 0;
  if (epi == EPI_STORE) {
    if (split) {
      if (vec) hipLaunchKernelGGL((ring_gemm_kernel<EPI_STORE, 1, true>), grid, dim3(NTHREADS), 0, s, gs);
      else hipLaunchKernelGGL((ring_gemm_kernel<EPI_STORE, 0, true>), grid, dim3(NTHREADS), 0, s, gs);
    } else {
      if (vec) hipLaunchKernelGGL((ring_gemm_kernel<EPI_STORE, 1, false>), grid, dim3(NTHREADS), 0, s, gs);
      else hipLaunchKernelGGL((ring_gemm_kernel<EPI_STORE, 0, false>), grid, dim3(NTHREADS), 0, s, gs);
    }
  } else if (epi == EPI_ACCUM) {
    if (split) {
      if (vec) hipLaunchKernelGGL((ring_gemm_kernel<EPI_ACCUM, 1, true>), grid, dim3(NTHREADS), 0, s, gs);
      else hipLaunchKernelGGL((ring_gemm_kernel<EPI_ACCUM, 0, true>), grid, dim3(NTHREADS), 0, s, gs);
    } else {
      if (vec) hipLaunchKernelGGL((ring_gemm_kernel<EPI_ACCUM, 1, false>), grid, dim3(NTHREADS), 0, s, gs);
      else hipLaunchKernelGGL((ring_gemm_kernel<EPI_ACCUM, 0, false>), grid, dim3(NTHREADS), 0, s, gs);
    }
  } else {
    if (vec) hipLaunchKernelGGL((ring_gemm_kernel<EPI_UNMASK, 1, false>), grid, dim3(NTHREADS), 0, s, gs);
    else hipLaunchKernelGGL((ring_gemm_kernel<EPI_UNMASK, 0, false>), grid, dim3(NTHREADS), 0, s, gs);
  }
  return hipGetLastError();
}

}  // namespace mosaic
