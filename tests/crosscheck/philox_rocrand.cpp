// Test-only cross-check: prints Philox-4x32-10 blocks from rocRAND's engine
// header (an implementation independent of the oracle's), host side only.
// Usage: philox_rocrand seed e nblocks. rocRAND's offset counts 32-bit
// values, so block b of epoch e is value offset 4 * ((e << 32) | b).
#include <rocrand/rocrand_philox4x32_10.h>
#include <cstdio>
#include <cstdlib>

int main(int argc, char** argv) {
  if (argc != 4) return 2;
  unsigned long long seed = std::strtoull(argv[1], nullptr, 10);
  unsigned long long e = std::strtoull(argv[2], nullptr, 10);
  long long nblocks = std::atoll(argv[3]);
  for (long long b = 0; b < nblocks; ++b) {
    rocrand_state_philox4x32_10 st;
    rocrand_init(seed, 0, 4ull * ((e << 32) | (unsigned long long)b), &st);
    unsigned w0 = rocrand(&st), w1 = rocrand(&st), w2 = rocrand(&st),
             w3 = rocrand(&st);
    std::printf("%u %u %u %u\n", w0, w1, w2, w3);
  }
  return 0;
}
