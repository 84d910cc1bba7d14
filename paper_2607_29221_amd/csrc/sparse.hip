// Sparse LPN matrices of the nested mask (Section 4.2 protocol box: S_{i+1}
// on the weight side, T_{i+1} on the activation side; LPN noise of rate
// 2^-s, Section 3) handled in compressed-row form, so that the client's
// products with them cost O(nonzeros) instead of the dense O(r_i) per output
// (the client-cost argument of Section 4.2 with Table "lpn-tradeoff").
//
// The matrices are the SPARSE streams of mosaic.h: element (i, j) of a
// rows x cols matrix is e = i cols + j, nonzero iff the top s bits of word 2e
// are zero, and then equal to word 2e + 1. Compressed rows list the nonzeros
// of each row in increasing column order. Or they are WEIGHT streams (the
// fixed Hamming weight t of Example 4.1): row i holds t entries chosen by a
// partial Fisher-Yates shuffle driven by words 2ti .. 2ti+2t-1, listed in
// the order of the shuffle's steps.
#include "internal.h"

namespace mosaic {
namespace {

// Entries of row ``row`` of a WEIGHT stream matrix, computed by one wave
// (the calling workgroup's first 64 threads; every thread of the workgroup
// must call it, the others only wait). scratch: weighted_scratch_bytes(cols,
// t) of LDS; pos / val (LDS, t entries) receive the chosen column and the
// value of each step. Ends with a workgroup barrier, after which pos and val
// are visible to all threads.
//
// Step j of the partial shuffle draws k_j = j + floor(u_j (cols - j) / 2^32)
// and swaps entries j and k_j of a running permutation (the identity at
// first); its column is the entry that lands at j, i.e. entry k_j just
// before the step. Up to WEIGHT_PAR_T steps that entry is found without
// running the swaps one after the other: position p >= j has been touched
// before step j only by the steps i < j with k_i = p (the steps' own
// positions i are all below j), and the latest of them left there the entry
// that position i held just before step i. Position i in turn held i unless
// an earlier step i' < i had k_{i'} = i, in which case it held what position
// i' held before step i', and so on. So the column of step j is k_j if no
// earlier step chose k_j, else E(i) for the latest such i, with E(i) = i if
// no step before i chose position i and E(i) = E(i') for the latest such i'.
// A table over the positions counts each position's choosers (and keeps
// the first one): a step whose position has one chooser takes it; the few
// steps on positions chosen more than once (a handful per row at t = 80 of
// r = 1024) go to a short list, which answers "latest earlier chooser" for
// them and, with the table, the chains of E. Longer rows take the steps one
// by one on a permutation kept in LDS as perm[k] ^ k, so that zero-filled
// memory is the identity.
constexpr int WEIGHT_PAR_T = 256;

inline size_t weighted_scratch_bytes(int64_t cols, int64_t t) {
  return t <= WEIGHT_PAR_T ? (size_t)(4 * cols + 8 * t + 16) : (size_t)(2 * cols + 4 * t + 16);
}

__device__ void weighted_row(const RngArgs& r, int64_t row, int cols, void* scratch, int32_t* pos, uint32_t* val) {
  const int t = r.row_weight;
  const int tid = threadIdx.x;
  const uint64_t w0 = 2 * (uint64_t)t * (uint64_t)row;   // even: each (u, value) pair is one half block
  if (t <= WEIGHT_PAR_T) {
    uint32_t* tab = (uint32_t*)scratch;        // per position: (choosers << 16) | first chooser
    uint32_t* kk = tab + cols;                 // per step: its position
    int32_t* shared_steps = (int32_t*)(kk + t); // steps on positions with several choosers
    int* nshared = (int*)(shared_steps + t);
    const int lane = tid;
    uint32_t k[4];
    if (tid < 64) {
      for (int p = lane; p < cols; p += 64) tab[p] = 0;
      if (lane == 0) *nshared = 0;
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        const int j = lane + 64 * s;
        k[s] = 0;
        if (j < t) {
          const uint64_t w = w0 + 2 * (uint64_t)j;
          const uint4 blk = philox_block(r, w >> 2);
          const bool hi = ((w >> 1) & 1) != 0;
          const uint32_t uj = hi ? blk.z : blk.x;
          val[j] = hi ? blk.w : blk.y;
          k[s] = (uint32_t)j + (uint32_t)(((uint64_t)uj * (uint64_t)(uint32_t)(cols - j)) >> 32);
          kk[j] = k[s];
        }
      }
    }
    __syncthreads();
    if (tid < 64) {
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        const int j = lane + 64 * s;
        if (j < t) {
          // the first chooser's step number goes to the low half; the others
          // only add to the count, so the two updates commute
          const uint32_t old = atomicAdd(&tab[k[s]], 0x10000u);
          if ((old >> 16) == 0) atomicOr(&tab[k[s]], (uint32_t)j);
        }
      }
    }
    __syncthreads();
    if (tid < 64) {
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        const int j = lane + 64 * s;
        if (j < t && (tab[k[s]] >> 16) >= 2) shared_steps[atomicAdd(nshared, 1)] = j;
      }
    }
    __syncthreads();
    if (tid < 64) {
      const int n = *nshared;
      // latest step before `before` whose position is p, or -1
      auto latest = [&](uint32_t p, int before) -> int {
        const uint32_t e = tab[p];
        const uint32_t choosers = e >> 16;
        if (choosers == 0) return -1;
        if (choosers == 1) return ((int)(e & 0xFFFFu) < before) ? (int)(e & 0xFFFFu) : -1;
        int best = -1;
        for (int q = 0; q < n; ++q) {
          const int i = shared_steps[q];
          if (i < before && i > best && kk[i] == p) best = i;
        }
        return best;
      };
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        const int j = lane + 64 * s;
        if (j < t) {
          int x = latest(k[s], j);
          uint32_t col = k[s];
          if (x >= 0) {
            for (int y = latest((uint32_t)x, x); y >= 0; y = latest((uint32_t)x, x)) x = y;
            col = (uint32_t)x;
          }
          pos[j] = (int32_t)col;
        }
      }
    }
    __syncthreads();
    return;
  }
  uint16_t* perm = (uint16_t*)scratch;
  uint32_t* u = (uint32_t*)scratch + ((cols + 1) >> 1);
  if (tid < 64) {
    for (int k = tid; k < cols; k += 64) perm[k] = 0;
    for (int j = tid; j < t; j += 64) {
      const uint64_t w = w0 + 2 * (uint64_t)j;
      const uint4 blk = philox_block(r, w >> 2);
      const bool hi = ((w >> 1) & 1) != 0;
      u[j] = hi ? blk.z : blk.x;
      val[j] = hi ? blk.w : blk.y;
    }
  }
  __syncthreads();
  if (tid == 0) {
    for (int j = 0; j < t; ++j) {
      const uint32_t k = (uint32_t)j + (uint32_t)(((uint64_t)u[j] * (uint64_t)(uint32_t)(cols - j)) >> 32);
      const uint32_t a = perm[j] ^ (uint32_t)j;     // entries j and k of the running permutation
      const uint32_t b = perm[k] ^ k;
      perm[j] = (uint16_t)(b ^ (uint32_t)j);
      perm[k] = (uint16_t)(a ^ k);
      pos[j] = (int32_t)b;
    }
  }
  __syncthreads();
}

// Dynamic LDS of the WEIGHT kernels: pos (t), val (t), then the row's
// scratch.
inline size_t weighted_lds_bytes(int64_t cols, int64_t t) { return (size_t)(8 * t) + weighted_scratch_bytes(cols, t); }

// One 64-thread workgroup per row: the row of a WEIGHT matrix as ring words
// and/or digits (zeros, then the t entries).
__global__ __launch_bounds__(64) void weighted_sample_kernel(RngArgs r, int64_t cols, uint32_t* out, int64_t ldo,
                                                             int8_t* dig, int64_t pitch) {
  extern __shared__ uint32_t wlds[];
  const int t = r.row_weight;
  int32_t* pos = (int32_t*)wlds;
  uint32_t* val = wlds + t;
  const int64_t row = blockIdx.x;
  const int tid = threadIdx.x;
  if (out != nullptr)
    for (int64_t k = tid; k < cols; k += 64) out[row * ldo + k] = 0u;
  if (dig != nullptr) {
    const int64_t bytes = 4 * (64 * ((cols + 63) / 64));   // the padded row, zero digits
    for (int64_t k = 16 * tid; k < bytes; k += 16 * 64) *(uint4*)(dig + row * pitch + k) = make_uint4(0, 0, 0, 0);
  }
  weighted_row(r, row, (int)cols, wlds + 2 * t, pos, val);   // its barriers also order the zero stores first
  for (int j = tid; j < t; j += 64) {
    const int64_t c = pos[j];
    const uint32_t v = val[j];
    if (out != nullptr) out[row * ldo + c] = v;
    if (dig != nullptr) {
      const uint32_t w = digit_word(v);
      int8_t* g = dig + row * pitch + 64 * (c >> 4) + (c & 15);
#pragma unroll
      for (int q = 0; q < 4; ++q) g[16 * q] = (int8_t)(w >> (8 * q));
    }
  }
}

// row_ptr[i] = i t for a WEIGHT matrix (rows + 1 entries).
__global__ __launch_bounds__(256) void weighted_count_kernel(int64_t rows, int64_t t, int64_t* row_ptr) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i <= rows) row_ptr[i] = i * t;
}

// One 64-thread workgroup per row: the row's t entries into its compressed
// row (at row_ptr[row]).
__global__ __launch_bounds__(64) void weighted_fill_kernel(RngArgs r, int64_t cols, const int64_t* row_ptr,
                                                           int32_t* col_idx, uint32_t* values) {
  extern __shared__ uint32_t wlds[];
  const int t = r.row_weight;
  const int64_t row = blockIdx.x;
  weighted_row(r, row, (int)cols, wlds + 2 * t, (int32_t*)wlds, wlds + t);
  const int64_t base = row_ptr[row];
  for (int j = threadIdx.x; j < t; j += 64) {
    col_idx[base + j] = (int32_t)wlds[j];
    values[base + j] = wlds[t + j];
  }
}

// gate and value of element e (words 2e and 2e + 1 share a Philox block)
__device__ __forceinline__ bool sparse_elem(const RngArgs& r, uint64_t e, uint32_t* val) {
  const uint4 blk = philox_block(r, e >> 1);
  const bool hi = (e & 1) != 0;
  const uint32_t gate = hi ? blk.z : blk.x;
  *val = hi ? blk.w : blk.y;
  return (r.sparse_shift >= 32) ? true : ((gate >> r.sparse_shift) == 0u);
}

// One wave per row: nonzero count of the row.
__global__ __launch_bounds__(256) void sparse_count_kernel(RngArgs r, int64_t rows, int64_t cols, int64_t* counts) {
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= rows) return;
  uint32_t n = 0, v;
  for (int64_t j = lane; j < cols; j += 64) n += sparse_elem(r, (uint64_t)row * cols + j, &v) ? 1u : 0u;
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) n += __shfl_xor(n, off);
  if (lane == 0) counts[row] = n;
}

// One workgroup: row_ptr[i] = sum of counts[0 .. i-1], row_ptr[rows] = total.
// counts and row_ptr may be the same array shifted by one (counts = row_ptr + 1).
__global__ __launch_bounds__(1024) void exclusive_scan_kernel(const int64_t* counts, int64_t rows, int64_t* row_ptr) {
  __shared__ int64_t part[1024];
  const int t = threadIdx.x;
  const int64_t per = (rows + 1023) / 1024;
  const int64_t b = t * per, e = (b + per < rows) ? b + per : rows;
  int64_t s = 0;
  for (int64_t i = b; i < e; ++i) s += counts[i];
  // When counts aliases row_ptr + 1, the neighbour's write of row_ptr[e]
  // overwrites counts[e - 1]: keep this chunk's last count in a register.
  const int64_t last = (e > b) ? counts[e - 1] : 0;
  part[t] = s;
  __syncthreads();
  for (int off = 1; off < 1024; off <<= 1) {       // inclusive Hillis-Steele scan of the chunk sums
    const int64_t add = (t >= off) ? part[t - off] : 0;
    __syncthreads();
    part[t] += add;
    __syncthreads();
  }
  int64_t run = (t > 0) ? part[t - 1] : 0;
  for (int64_t i = b; i < e; ++i) {                  // counts[i] is read before row_ptr[i] (= counts[i-1]) moves
    const int64_t c = (i == e - 1) ? last : counts[i];
    row_ptr[i] = run;
    run += c;
  }
  if (t == 1023) row_ptr[rows] = part[1023];
}

// One wave per row: nonzeros written in column order (ballot + prefix count).
__global__ __launch_bounds__(256) void sparse_fill_kernel(RngArgs r, int64_t rows, int64_t cols,
                                                          const int64_t* row_ptr, int32_t* col_idx, uint32_t* values) {
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= rows) return;
  int64_t base = row_ptr[row];
  for (int64_t j0 = 0; j0 < cols; j0 += 64) {
    const int64_t j = j0 + lane;
    uint32_t v = 0;
    const bool nz = (j < cols) && sparse_elem(r, (uint64_t)row * cols + j, &v);
    const uint64_t mask = __ballot(nz);
    if (nz) {
      const int64_t pos = base + __popcll(mask & ((1ull << lane) - 1ull));
      col_idx[pos] = (int32_t)j;
      values[pos] = v;
    }
    base += __popcll(mask);
  }
}

// c[i][k] +-= sum_j P(i, j) d[j][k] for k < ncols. A workgroup owns
// 256 / NSPLIT consecutive k of one row i. The row's nonzeros are staged in LDS in chunks
// of CH entries -- copied from compressed rows (STREAM = 0), drawn from the
// SPARSE stream of rng over the row's rcols columns (STREAM = 1: each wave
// appends its nonzeros through an LDS counter; the ring sum does not depend
// on their order) or drawn as the t entries of a WEIGHT row (STREAM = 2, one
// chunk: t <= CH; the shuffle's scratch is dynamic LDS). Each lane takes one
// k, so a load instruction reads 256 consecutive bytes of a row of d; the
// NSPLIT waves that share 64 k split the staged entries (wave w takes
// entries w % NSPLIT, + NSPLIT, ..., LDS broadcasts) and their partial sums
// meet in LDS. NSPLIT = 4 gives rows with few workgroups four times as many
// (one token against an 8192-column d: 128 instead of 32 workgroups, 8.4 us
// before); with many rows NSPLIT = 1 keeps the per-workgroup staging (for a
// WEIGHT row, a serial shuffle) from being repeated four times as often.
template <int STREAM, int NSPLIT>
__global__ __launch_bounds__(256) void gather_rows_kernel(RngArgs r, int64_t rcols, const int64_t* row_ptr,
                                                          const int32_t* col_idx, const uint32_t* values,
                                                          const uint32_t* d, int64_t ldd, int64_t ncols,
                                                          uint32_t* c, int64_t ldc, int subtract) {
  constexpr int CH = 2048;
  __shared__ int32_t scol[CH];
  __shared__ uint32_t sval[CH];
  __shared__ uint32_t part[4][64];
  __shared__ int scount;
  static_assert(NSPLIT == 1 || NSPLIT == 2 || NSPLIT == 4, "waves per column group");
  const int tid = threadIdx.x;
  const int wave = tid >> 6;
  const int64_t i = blockIdx.x;
  const int64_t k = (int64_t)blockIdx.y * (256 / NSPLIT) + (wave / NSPLIT) * 64 + (tid & 63);
  const bool active = k < ncols;
  const uint32_t* dk = d + (active ? k : 0);
  const int64_t lo = STREAM ? 0 : row_ptr[i];
  const int64_t hi = STREAM == 2 ? r.row_weight : STREAM ? rcols : row_ptr[i + 1];
  uint32_t acc = 0;
  for (int64_t base = lo; base < hi; base += CH) {
    const int64_t end = (base + CH < hi) ? base + CH : hi;
    int n;
    if (STREAM == 2) {
      extern __shared__ uint32_t wlds[];
      weighted_row(r, i, (int)rcols, wlds, scol, sval);
      n = r.row_weight;
    } else if (STREAM == 1) {
      if (tid == 0) scount = 0;
      __syncthreads();
      for (int64_t j0 = base; j0 < end; j0 += 256) {
        const int64_t j = j0 + tid;
        uint32_t v = 0;
        const bool nz = (j < end) && sparse_elem(r, (uint64_t)i * rcols + j, &v);
        const uint64_t mask = __ballot(nz);
        const int lane = tid & 63;
        int wbase = 0;
        if (lane == 0 && mask) wbase = atomicAdd(&scount, __popcll(mask));
        wbase = __shfl(wbase, 0);
        if (nz) {
          const int pos = wbase + __popcll(mask & ((1ull << lane) - 1ull));
          scol[pos] = (int32_t)j;
          sval[pos] = v;
        }
      }
      __syncthreads();
      n = scount;
    } else {
      for (int64_t p = base + tid; p < end; p += 256) {
        scol[p - base] = col_idx[p];
        sval[p - base] = values[p];
      }
      __syncthreads();
      n = (int)(end - base);
    }
    if (active) {
      constexpr int ST = NSPLIT;
      int q = wave % NSPLIT;
      for (; q + 3 * ST < n; q += 4 * ST) {
        const uint32_t a0 = dk[(int64_t)scol[q] * ldd], a1 = dk[(int64_t)scol[q + ST] * ldd];
        const uint32_t a2 = dk[(int64_t)scol[q + 2 * ST] * ldd], a3 = dk[(int64_t)scol[q + 3 * ST] * ldd];
        acc += sval[q] * a0 + sval[q + ST] * a1 + sval[q + 2 * ST] * a2 + sval[q + 3 * ST] * a3;
      }
      for (; q < n; q += ST) acc += sval[q] * dk[(int64_t)scol[q] * ldd];
    }
    __syncthreads();                                   // before the next chunk overwrites the staging
  }
  if (NSPLIT > 1) {
    part[wave][tid & 63] = acc;
    __syncthreads();
    if (wave % NSPLIT != 0) return;
#pragma unroll
    for (int w = 1; w < NSPLIT; ++w) acc += part[wave + w][tid & 63];
  }
  if (active) {
    uint32_t* out = c + i * ldc + k;
    *out = subtract ? *out - acc : *out + acc;
  }
}

// Waves per 64 columns of the row gathers: split a row's entries between
// four waves while that keeps the workgroup count under four per compute
// unit, else one wave per 64 columns.
int gather_split(int64_t rows, int64_t ncols) {
  return rows * ((ncols + 63) / 64) <= 4 * (int64_t)compute_units() ? 4 : 1;
}

// c[m][n] +-= sum_{p in row n} values[p] * d[m][col_idx[p]]. A workgroup owns
// 32 consecutive n and MB consecutive m; eight lanes share each n and split
// its nonzeros, so a row's entries are read once, in a few coalesced rounds,
// for MB rows of d (with one m per workgroup, 8 tokens against a 14336-row P
// with 80 entries per row re-read the entries 8 times: 23-25 us), then the
// eight partial sums of each m are combined with lane shuffles.
template <int MB>
__global__ __launch_bounds__(256) void gather_cols_kernel(int64_t M, int64_t N, const int64_t* row_ptr,
                                                          const int32_t* col_idx, const uint32_t* values,
                                                          const uint32_t* d, int64_t ldd, uint32_t* c, int64_t ldc,
                                                          int subtract, Dequant dq) {
  const int64_t m0 = (int64_t)blockIdx.x * MB;
  const int sub = threadIdx.x & 7;
  const int64_t n = (int64_t)blockIdx.y * 32 + (threadIdx.x >> 3);
  uint32_t acc[MB];
#pragma unroll
  for (int mm = 0; mm < MB; ++mm) acc[mm] = 0;
  if (n < N) {
    const int64_t p0 = row_ptr[n], p1 = row_ptr[n + 1];
    int64_t p = p0 + sub;
    // four of the lane's entries in flight at once (one at a time, each
    // entry's loads and then its gather from d waited in turn: one-token
    // calls over 14336 rows of 80 entries took 6.9 instead of 4.8 us)
    for (; p + 24 < p1; p += 32) {
      uint32_t v[4];
      int64_t col[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        v[q] = values[p + 8 * q];
        col[q] = col_idx[p + 8 * q];
      }
#pragma unroll
      for (int mm = 0; mm < MB; ++mm)
        if (m0 + mm < M) {
          const uint32_t* dr = d + (m0 + mm) * ldd;
          acc[mm] += v[0] * dr[col[0]] + v[1] * dr[col[1]] + v[2] * dr[col[2]] + v[3] * dr[col[3]];
        }
    }
    for (; p < p1; p += 8) {
      const uint32_t v = values[p];
      const int64_t col = col_idx[p];
#pragma unroll
      for (int mm = 0; mm < MB; ++mm)
        if (m0 + mm < M) acc[mm] += v * d[(m0 + mm) * ldd + col];
    }
  }
#pragma unroll
  for (int mm = 0; mm < MB; ++mm) {
    uint32_t a = acc[mm];
    a += __shfl_xor(a, 4, 8);
    a += __shfl_xor(a, 2, 8);
    a += __shfl_xor(a, 1, 8);
    const int64_t m = m0 + mm;
    if (n < N && sub == 0 && m < M) {
      uint32_t* out = c + m * ldc + n;
      const uint32_t val = subtract ? *out - a : *out + a;
      *out = val;
      if (dq.y != nullptr) {
        // the same steps and roundings as the unmask epilogue's dequantisation
        const float f = (float)(int32_t)val * dq.s_rows[m] * dq.s_cols[n];
        dq.y[m * dq.ld + n] = dq.bias != nullptr ? __fadd_rn(f, dq.bias[n]) : f;
      }
    }
  }
}

}  // namespace

hipError_t launch_sparse_csr_count(const RngArgs& r, int64_t rows, int64_t cols, int64_t* row_ptr, hipStream_t s) {
  // per-row counts land in row_ptr[1 ..], then the scan rewrites the array
  if (rows > 0)
    hipLaunchKernelGGL(sparse_count_kernel, dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, s, r, rows, cols,
                       row_ptr + 1);
  hipLaunchKernelGGL(exclusive_scan_kernel, dim3(1), dim3(1024), 0, s, row_ptr + 1, rows, row_ptr);
  return hipGetLastError();
}

hipError_t launch_sparse_csr_fill(const RngArgs& r, int64_t rows, int64_t cols, const int64_t* row_ptr,
                                  int32_t* col_idx, uint32_t* values, hipStream_t s) {
  if (rows == 0) return hipSuccess;
  hipLaunchKernelGGL(sparse_fill_kernel, dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, s, r, rows, cols, row_ptr,
                     col_idx, values);
  return hipGetLastError();
}

hipError_t launch_sparse_gather_rows(int64_t rows, const int64_t* row_ptr, const int32_t* col_idx,
                                     const uint32_t* values, const uint32_t* d, int64_t ldd, int64_t ncols,
                                     uint32_t* c, int64_t ldc, int subtract, hipStream_t s) {
  if (rows == 0 || ncols == 0) return hipSuccess;
  if (gather_split(rows, ncols) == 4)
    hipLaunchKernelGGL((gather_rows_kernel<0, 4>), dim3((unsigned)rows, (unsigned)((ncols + 63) / 64)), dim3(256), 0,
                       s, RngArgs{}, (int64_t)0, row_ptr, col_idx, values, d, ldd, ncols, c, ldc, subtract);
  else
    hipLaunchKernelGGL((gather_rows_kernel<0, 1>), dim3((unsigned)rows, (unsigned)((ncols + 255) / 256)), dim3(256),
                       0, s, RngArgs{}, (int64_t)0, row_ptr, col_idx, values, d, ldd, ncols, c, ldc, subtract);
  return hipGetLastError();
}

hipError_t launch_sparse_stream_gather_rows(const RngArgs& r, int64_t rows, int64_t rcols, const uint32_t* d,
                                            int64_t ldd, int64_t ncols, uint32_t* c, int64_t ldc, int subtract,
                                            hipStream_t s) {
  if (rows == 0 || ncols == 0 || rcols == 0) return hipSuccess;
  const bool split = gather_split(rows, ncols) == 4;
  const dim3 grid((unsigned)rows, (unsigned)(split ? (ncols + 63) / 64 : (ncols + 255) / 256));
  const int64_t* np = nullptr;
  const int32_t* ni = nullptr;
  const uint32_t* nv = nullptr;
  if (r.dist == 4) {
    if (r.row_weight == 0) return hipSuccess;
    // the drawn row's scratch; its entries go to the static staging arrays
    const size_t lds = weighted_scratch_bytes(rcols, r.row_weight);
    if (split)
      hipLaunchKernelGGL((gather_rows_kernel<2, 4>), grid, dim3(256), lds, s, r, rcols, np, ni, nv, d, ldd, ncols, c,
                         ldc, subtract);
    else
      hipLaunchKernelGGL((gather_rows_kernel<2, 1>), grid, dim3(256), lds, s, r, rcols, np, ni, nv, d, ldd, ncols, c,
                         ldc, subtract);
  } else {
    if (split)
      hipLaunchKernelGGL((gather_rows_kernel<1, 4>), grid, dim3(256), 0, s, r, rcols, np, ni, nv, d, ldd, ncols, c,
                         ldc, subtract);
    else
      hipLaunchKernelGGL((gather_rows_kernel<1, 1>), grid, dim3(256), 0, s, r, rcols, np, ni, nv, d, ldd, ncols, c,
                         ldc, subtract);
  }
  return hipGetLastError();
}

hipError_t launch_weighted_sample(const RngArgs& r, int64_t rows, int64_t cols, uint32_t* out, int64_t ldo,
                                  int8_t* dig, int64_t pitch, hipStream_t s) {
  if (rows == 0 || cols == 0) return hipSuccess;
  hipLaunchKernelGGL(weighted_sample_kernel, dim3((unsigned)rows), dim3(64), weighted_lds_bytes(cols, r.row_weight), s,
                     r, cols, out, ldo, dig, pitch);
  return hipGetLastError();
}

hipError_t launch_weighted_csr_count(int64_t rows, int64_t t, int64_t* row_ptr, hipStream_t s) {
  hipLaunchKernelGGL(weighted_count_kernel, dim3((unsigned)((rows + 1 + 255) / 256)), dim3(256), 0, s, rows, t,
                     row_ptr);
  return hipGetLastError();
}

hipError_t launch_weighted_csr_fill(const RngArgs& r, int64_t rows, int64_t cols, const int64_t* row_ptr,
                                    int32_t* col_idx, uint32_t* values, hipStream_t s) {
  if (rows == 0 || cols == 0 || r.row_weight == 0) return hipSuccess;
  hipLaunchKernelGGL(weighted_fill_kernel, dim3((unsigned)rows), dim3(64), weighted_lds_bytes(cols, r.row_weight), s,
                     r, cols, row_ptr, col_idx, values);
  return hipGetLastError();
}

hipError_t launch_sparse_gather_cols(int64_t M, int64_t N, const int64_t* row_ptr, const int32_t* col_idx,
                                     const uint32_t* values, const uint32_t* d, int64_t ldd, uint32_t* c,
                                     int64_t ldc, int subtract, const Dequant& dq, hipStream_t s) {
  if (M == 0 || N == 0) return hipSuccess;
  const unsigned nb = (unsigned)((N + 31) / 32);
  // rows of d per workgroup: as many as keep four workgroups per compute
  // unit (up to 16), so that a row's entries are read fewer times without
  // losing the parallelism the short rows need
  int mb = 1;
  while (mb < 16 && mb < M && ((M + 2 * mb - 1) / (2 * mb)) * (int64_t)nb >= 4 * (int64_t)compute_units()) mb *= 2;
  const dim3 grid((unsigned)((M + mb - 1) / mb), nb);
  switch (mb) {
    case 1: hipLaunchKernelGGL((gather_cols_kernel<1>), grid, dim3(256), 0, s, M, N, row_ptr, col_idx, values, d,
                               ldd, c, ldc, subtract, dq); break;
    case 2: hipLaunchKernelGGL((gather_cols_kernel<2>), grid, dim3(256), 0, s, M, N, row_ptr, col_idx, values, d,
                               ldd, c, ldc, subtract, dq); break;
    case 4: hipLaunchKernelGGL((gather_cols_kernel<4>), grid, dim3(256), 0, s, M, N, row_ptr, col_idx, values, d,
                               ldd, c, ldc, subtract, dq); break;
    case 8: hipLaunchKernelGGL((gather_cols_kernel<8>), grid, dim3(256), 0, s, M, N, row_ptr, col_idx, values, d,
                               ldd, c, ldc, subtract, dq); break;
    default: hipLaunchKernelGGL((gather_cols_kernel<16>), grid, dim3(256), 0, s, M, N, row_ptr, col_idx, values, d,
                                ldd, c, ldc, subtract, dq); break;
  }
  return hipGetLastError();
}

}  // namespace mosaic
