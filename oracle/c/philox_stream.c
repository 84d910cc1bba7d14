/*
 * Oracle (test infrastructure): bulk Philox-4x32-10 stream words in plain C,
 * for the full-size sampled checks. Same definition as oracle/philox.py
 * (Salmon, Moraes, Dror, Shaw, SC'11): ten rounds of
 *   (c0, c1, c2, c3) -> (hi(M1 c2) ^ c1 ^ k0, lo(M1 c2), hi(M0 c0) ^ c3 ^ k1, lo(M0 c0))
 * with the key advanced by the Weyl increments between rounds.
 * Stream word t is word (t mod 4) of the block with counter
 * (b mod 2^32, b div 2^32, stream, instance), b = t div 4, and key
 * (seed mod 2^32, seed div 2^32).
 */
#include <stdint.h>

static void philox_block(uint64_t b, uint32_t stream, uint32_t instance, uint32_t k0, uint32_t k1,
                         uint32_t out[4]) {
  uint32_t c0 = (uint32_t)b, c1 = (uint32_t)(b >> 32), c2 = stream, c3 = instance;
  for (int r = 0; r < 10; ++r) {
    const uint64_t p0 = (uint64_t)0xD2511F53u * c0;
    const uint64_t p1 = (uint64_t)0xCD9E8D57u * c2;
    const uint32_t n0 = (uint32_t)(p1 >> 32) ^ c1 ^ k0;
    const uint32_t n1 = (uint32_t)p1;
    const uint32_t n2 = (uint32_t)(p0 >> 32) ^ c3 ^ k1;
    const uint32_t n3 = (uint32_t)p0;
    c0 = n0; c1 = n1; c2 = n2; c3 = n3;
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
  out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

/* words t0 .. t0 + count - 1 of stream (seed, stream, instance); ranges of
 * words are independent, so OpenMP threads take consecutive slices */
void oracle_stream_words(uint64_t seed, uint32_t stream, uint32_t instance, uint64_t t0, uint64_t count,
                         uint32_t* out) {
  const uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
  const int64_t slices = (int64_t)((count + 65535) >> 16);
#pragma omp parallel for schedule(static)
  for (int64_t sl = 0; sl < slices; ++sl) {
    const uint64_t i0 = (uint64_t)sl << 16;
    const uint64_t i1 = (i0 + 65536 < count) ? i0 + 65536 : count;
    uint32_t blk[4];
    uint64_t have = ~(uint64_t)0;
    for (uint64_t i = i0; i < i1; ++i) {
      const uint64_t t = t0 + i;
      const uint64_t b = t >> 2;
      if (b != have) {
        philox_block(b, stream, instance, k0, k1, blk);
        have = b;
      }
      out[i] = blk[t & 3];
    }
  }
}
