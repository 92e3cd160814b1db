// Philox4x32-10 blocks from rocRAND's engine (test infrastructure: an
// implementation of the generator that is independent of the oracle's).
// Reads lines "c0 c1 c2 c3 k0 k1" (decimal uint32) from stdin and prints the
// four output words of each block.
#include <rocrand/rocrand_philox4x32_10.h>

#include <cstdio>

namespace {

struct Block : rocrand_device::philox4x32_10_engine {
  uint4 run(uint4 counter, uint2 key) { return ten_rounds(counter, key); }
};

}  // namespace

int main() {
  Block b;
  unsigned c0, c1, c2, c3, k0, k1;
  while (std::scanf("%u %u %u %u %u %u", &c0, &c1, &c2, &c3, &k0, &k1) == 6) {
    const uint4 r = b.run(uint4{c0, c1, c2, c3}, uint2{k0, k1});
    std::printf("%u %u %u %u\n", r.x, r.y, r.z, r.w);
  }
  return 0;
}
