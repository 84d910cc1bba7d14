// Device helpers shared by the MOSAIC kernels: the Philox-4x32-10 generator,
// the mask-material samplers and the signed-digit form of ring elements.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mosaic {

constexpr int kMaxDgaussBound = 15;

// 16-byte vectors for __builtin_nontemporal_load/store, which stream data
// that a kernel reads or writes once.
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Parameters of one random stream as the kernels see them (passed by value).
struct RngArgs {
  uint32_t k0, k1;        // Philox key: seed low / high word
  uint32_t stream;        // counter word 2
  uint32_t instance;      // counter word 3
  int32_t dist;           // mosaic_dist
  int32_t bound;          // DGAUSS support [-bound, bound]
  int32_t sparse_shift;   // SPARSE: 32 - s (gate kept when gate >> shift == 0); 32 keeps all
  int32_t transposed;
  int32_t row_weight;     // WEIGHT: entries per row
  // DGAUSS inverse-CDF table. Of the 2 bound thresholds T_k (ascending, in
  // [0, 2^32]) those equal to 0 count for every word and those equal to 2^32
  // for none: they are folded into dg_base = -bound + #{T_k = 0}; the
  // dg_count others lie strictly inside (0, 2^32) and fit in 32 bits.
  int32_t dg_base;
  int32_t dg_count;
  uint32_t th[2 * kMaxDgaussBound];
};

// Philox-4x32 with 10 rounds (Salmon et al., SC'11): each round multiplies
// words 0 and 2 by fixed odd constants into 64-bit products and outputs
// (hi(M1 c2) ^ c1 ^ k0, lo(M1 c2), hi(M0 c0) ^ c3 ^ k1, lo(M0 c0)); the key
// advances by the Weyl increments between rounds.
// a ^ b ^ k in one instruction: gfx950's three-input bitwise operation with
// truth table 0x96 (odd parity of the three bits); the compiler emits two
// two-input XORs for the expression. k is uniform (a Philox key word, in a
// scalar register: one scalar operand per vector instruction).
__device__ __forceinline__ uint32_t xor3(uint32_t a, uint32_t b, uint32_t k) {
  uint32_t r;
  asm("v_bitop3_b32 %0, %1, %2, %3 bitop3:0x96" : "=v"(r) : "v"(a), "v"(b), "s"(k));
  return r;
}

__device__ __forceinline__ uint4 philox4x32_10(uint4 c, uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    const uint64_t p0 = (uint64_t)0xD2511F53u * c.x;
    const uint64_t p1 = (uint64_t)0xCD9E8D57u * c.z;
    const uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
    const uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
    c = make_uint4(xor3(hi1, c.y, k0), lo1, xor3(hi0, c.w, k1), lo0);
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
  return c;
}

__device__ __forceinline__ uint4 philox_block(const RngArgs& r, uint64_t b) {
  return philox4x32_10(make_uint4((uint32_t)b, (uint32_t)(b >> 32), r.stream, r.instance), r.k0, r.k1);
}

__device__ __forceinline__ uint32_t pick(const uint4& v, uint32_t lane) {
  return lane == 0 ? v.x : lane == 1 ? v.y : lane == 2 ? v.z : v.w;
}

__device__ __forceinline__ uint32_t stream_word(const RngArgs& r, uint64_t t) {
  return pick(philox_block(r, t >> 2), (uint32_t)(t & 3));
}

__device__ __forceinline__ uint32_t dgauss_from_word(const RngArgs& r, uint32_t u) {
  int32_t v = r.dg_base;
  for (int k = 0; k < r.dg_count; ++k) v += (u >= r.th[k]) ? 1 : 0;
  return (uint32_t)v;
}

// The same for four words at once. For 0 < T < 2^32, u >= T exactly when
// u + (2^32 - T) carries out of 32 bits, so the count advances by the carry
// of that add (an add and an add-with-carry, no compare); an addend of 0
// never carries, which switches off the slots past dg_count. The first
// kDgaussInline slots are read at constant indices (scalar registers shared
// by the four words): six, the inner thresholds of sigma = 0.5 on [-4, 4];
// longer tables continue in the loop below. A loop over the table with a
// run-time index had read one threshold from memory per iteration and word
// and waited for it (the noisy mask pass took 134-147 us against 122 us
// with eight inline slots at 2048 x 28672).
constexpr int kDgaussInline = 6;
__device__ __forceinline__ void dgauss4(const RngArgs& r, uint32_t u[4]) {
  uint32_t v[4] = {(uint32_t)r.dg_base, (uint32_t)r.dg_base, (uint32_t)r.dg_base, (uint32_t)r.dg_base};
#pragma unroll
  for (int k = 0; k < kDgaussInline; ++k) {
    const uint32_t neg = k < r.dg_count ? 0u - r.th[k] : 0u;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      uint32_t lo;
      v[i] += __builtin_add_overflow(u[i], neg, &lo) ? 1u : 0u;
    }
  }
  for (int k = kDgaussInline; k < r.dg_count; ++k) {
    const uint32_t neg = 0u - r.th[k];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      uint32_t lo;
      v[i] += __builtin_add_overflow(u[i], neg, &lo) ? 1u : 0u;
    }
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) u[i] = v[i];
}

__device__ __forceinline__ uint32_t sparse_from_words(const RngArgs& r, uint32_t gate, uint32_t val) {
  const bool keep = (r.sparse_shift >= 32) ? true : ((gate >> r.sparse_shift) == 0u);
  return keep ? val : 0u;
}

// Element e of the stream's matrix (any alignment).
__device__ __forceinline__ uint32_t sample_elem(const RngArgs& r, uint64_t e) {
  switch (r.dist) {
    case 1: return stream_word(r, e);
    case 2: return dgauss_from_word(r, stream_word(r, e));
    case 3: {
      const uint4 blk = philox_block(r, (2 * e) >> 2);   // words 2e, 2e+1 share a block
      const uint32_t lane = (uint32_t)((2 * e) & 3);
      return sparse_from_words(r, pick(blk, lane), pick(blk, lane + 1));
    }
    default: return 0u;
  }
}

// Elements e0 .. e0+3 with e0 a multiple of 4: one Philox block (two for SPARSE).
__device__ __forceinline__ void sample4_aligned(const RngArgs& r, uint64_t e0, uint32_t out[4]) {
  if (r.dist == 1 || r.dist == 2) {
    const uint4 w = philox_block(r, e0 >> 2);
    out[0] = w.x; out[1] = w.y; out[2] = w.z; out[3] = w.w;
    if (r.dist == 2) dgauss4(r, out);
  } else if (r.dist == 3) {
    const uint4 a = philox_block(r, (2 * e0) >> 2);
    const uint4 b = philox_block(r, ((2 * e0) >> 2) + 1);
    out[0] = sparse_from_words(r, a.x, a.y);
    out[1] = sparse_from_words(r, a.z, a.w);
    out[2] = sparse_from_words(r, b.x, b.y);
    out[3] = sparse_from_words(r, b.z, b.w);
  } else {
    out[0] = out[1] = out[2] = out[3] = 0u;
  }
}

// Balanced base-256 digits of x packed in one word: byte t is digit t as an
// int8. Adding 0x80 to every byte position maps each balanced digit d to the
// ordinary byte d + 128 of x + 0x80808080; flipping bit 7 of every byte
// subtracts the 128 again in two's complement.
__device__ __forceinline__ uint32_t digit_word(uint32_t x) {
  return (x + 0x80808080u) ^ 0x80808080u;
}

// Transpose four digit words (elements k..k+3) into four words holding digit
// t of those four elements (byte b = element k+b): two rounds of byte
// permutes (__builtin_amdgcn_perm(hi, lo, sel): selector bytes 0-3 pick lo's
// bytes, 4-7 hi's), eight instructions for the 16 bytes.
__device__ __forceinline__ void digit_transpose4(const uint32_t w[4], uint32_t out[4]) {
  const uint32_t e01 = __builtin_amdgcn_perm(w[1], w[0], 0x06020400u);   // w0.0 w1.0 w0.2 w1.2
  const uint32_t o01 = __builtin_amdgcn_perm(w[1], w[0], 0x07030501u);   // w0.1 w1.1 w0.3 w1.3
  const uint32_t e23 = __builtin_amdgcn_perm(w[3], w[2], 0x06020400u);
  const uint32_t o23 = __builtin_amdgcn_perm(w[3], w[2], 0x07030501u);
  out[0] = __builtin_amdgcn_perm(e23, e01, 0x05040100u);
  out[1] = __builtin_amdgcn_perm(o23, o01, 0x05040100u);
  out[2] = __builtin_amdgcn_perm(e23, e01, 0x07060302u);
  out[3] = __builtin_amdgcn_perm(o23, o01, 0x07060302u);
}

// Digit planes of four consecutive ring elements: out[t] holds digit t of
// v[0..3] (byte b = element b).
__device__ __forceinline__ void digit_planes4(const uint32_t v[4], uint32_t out[4]) {
  const uint32_t w[4] = {digit_word(v[0]), digit_word(v[1]), digit_word(v[2]), digit_word(v[3])};
  digit_transpose4(w, out);
}

// Digit planes of one 16-column group held by four consecutive lanes: lane
// q of the quad holds ring values v[0..3] of columns 4 q .. 4 q + 3 and
// receives in o[0..3] the 16 bytes of digit plane q of the whole group
// (byte 4 r + b = digit q of column 4 r + b), i.e. the 16-byte word it stores
// at offset 16 q of the group's 64 bytes. Every lane of the quad must call it.
__device__ __forceinline__ void quad_digit_planes(const uint32_t v[4], int q, uint32_t o[4]) {
  const uint32_t w[4] = {digit_word(v[0]), digit_word(v[1]), digit_word(v[2]), digit_word(v[3])};
  uint32_t p[4];                                  // p[t]: digit t of this lane's 4 columns
  digit_transpose4(w, p);
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int src_t = q ^ r;                      // what this lane sends to lane q ^ r
    const uint32_t send = src_t == 0 ? p[0] : src_t == 1 ? p[1] : src_t == 2 ? p[2] : p[3];
    const uint32_t got = (r == 0) ? send : (uint32_t)__shfl_xor((int)send, r, 4);
    o[q ^ r] = got;                               // from lane q ^ r: its digit plane q
  }
}

// Quantised codes without a division per entry. The code of an entry is
// rint(fl(y / s)) (ties to even) with y = fl(v c) for a factor c of the
// entry and a row scale s with |y| <= qmax s up to the rounding of s, so
// |y / s| < L = qmax + 1. With r = fl(1 / s) and k = fl(c r), t = fl(v k)
// equals y / s up to four roundings of relative size u = 2^-24 (r, k, t and
// y): |t - y / s| <= (4 u + 8 u^2) |y / s|; fl(y / s) is within u |y / s|
// of it, so |t - fl(y / s)| < 6 u L. rint of t and of fl(y / s) can
// therefore differ only where a half-integer lies within 6 u L of t, i.e.
// where |t - rint(t)| > 1/2 - 6 u L; those entries (a fraction 12 u L of
// them) are computed by the division itself, and so are non-finite t.
// quant_threshold gives that bound, or -1 (every entry divides) where the
// argument needs more care: qmax >= 2^20, or s outside [2^-100, 2^100], which
// keeps r and k normal and the rounding of subnormal y far below the margin.
__device__ __forceinline__ float quant_threshold(float s, int32_t qmax) {
  const bool ok = s >= 0x1p-100f && s <= 0x1p100f && qmax < (1 << 20);
  return ok ? 0.5f - (float)(qmax + 1) * 0x1.8p-22f : -1.0f;   // 6 u L, exact in fp32
}

// Codes of four entries v[0..3] with a common factor c: k = fl(c fl(1 / s)),
// thr = quant_threshold(s, qmax). The codes equal rint(fl(fl(v c) / s)).
// One branch per entry: a wave runs a division only for an entry that one
// of its lanes needs. (One branch for all four entries, with a margin of
// 8 u L, sent 13-39% of the wave-groups of four entries through four
// divisions at qmax = 567-1997; the fused input pass was 1-10% slower.)
__device__ __forceinline__ void quant_codes4(const float v[4], float c, float k, float s, float thr,
                                             uint32_t q[4]) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float t = __fmul_rn(v[i], k);
    float f = rintf(t);
    if (!(fabsf(t - f) <= thr)) {
      // the divisor passes through an empty volatile statement, so that the
      // division stays inside this rarely taken branch
      float sd = s;
      asm volatile("" : "+v"(sd));
      f = rintf((v[i] * c) / sd);
    }
    q[i] = (uint32_t)(int32_t)f;
  }
}
}  // namespace mosaic
