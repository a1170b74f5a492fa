// Independent Philox4x32-10 reference for the oracle's tests: rocRAND's
// host-callable engine.  Reads lines "seed c0 c1 c2 c3" (hex or decimal) on
// stdin and prints the four output words of the block at counter
// (c0, c1, c2, c3) under key = seed.
#include <rocrand/rocrand_philox4x32_10.h>
#include <cstdio>
#include <cstdlib>

int main() {
  unsigned long long seed, c0, c1, c2, c3;
  while (std::scanf("%llx %llx %llx %llx %llx", &seed, &c0, &c1, &c2, &c3) == 5) {
    unsigned long long sub = c2 | (c3 << 32);
    rocrand_device::philox4x32_10_engine e(seed, sub, 0);
    unsigned long long n = c0 | (c1 << 32);          // blocks to skip
    const unsigned long long step = 1ull << 60;       // blocks per discard call
    while (n >= step) { e.discard(4ull * step); n -= step; }
    e.discard(4ull * n);
    uint4 r = e.next4();
    std::printf("%08x %08x %08x %08x\n", r.x, r.y, r.z, r.w);
  }
  return 0;
}
