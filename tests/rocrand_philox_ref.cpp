// Reference Philox-4x32-10 for the oracle's pin: reads lines of
// "c0 c1 c2 c3 k0 k1" (decimal 32-bit words) and prints the four output words
// of rocRAND's Philox-4x32-10 block function for that counter and key. Built
// and run on the host by tests/test_oracle_philox.py; rocRAND's header is
// independent open source (Random123's constants and round), not part of this
// repository's device code.
#include <rocrand/rocrand_philox4x32_10.h>
#include <cstdio>

namespace {
struct Block : rocrand_device::philox4x32_10_engine {
  using rocrand_device::philox4x32_10_engine::ten_rounds;
};
}  // namespace

int main() {
  unsigned c0, c1, c2, c3, k0, k1;
  Block eng;
  while (std::scanf("%u %u %u %u %u %u", &c0, &c1, &c2, &c3, &k0, &k1) == 6) {
    const uint4 r = eng.ten_rounds(uint4{c0, c1, c2, c3}, uint2{k0, k1});
    std::printf("%u %u %u %u\n", r.x, r.y, r.z, r.w);
  }
  return 0;
}
