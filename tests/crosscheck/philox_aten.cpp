// Test-only cross-check: prints Philox-4x32-10 blocks from PyTorch's own
// engine header (an implementation independent of the oracle's), for
// counters (k/4, e, 0, 0) and key (seed lo, seed hi). Reads "seed e nblocks"
// on the command line and prints one line of four words per block.
#include <ATen/core/PhiloxRNGEngine.h>
#include <cstdio>
#include <cstdlib>

int main(int argc, char** argv) {
  if (argc != 4) return 2;
  unsigned long long seed = std::strtoull(argv[1], nullptr, 10);
  unsigned long long e = std::strtoull(argv[2], nullptr, 10);
  long long nblocks = std::atoll(argv[3]);
  for (long long b = 0; b < nblocks; ++b) {
    // offset = (e << 32) | b puts b in counter word 0 and e in word 1;
    // subsequence 0 leaves words 2 and 3 at zero.
    at::Philox4_32 eng(seed, 0, (e << 32) | (unsigned long long)b);
    unsigned w0 = eng(), w1 = eng(), w2 = eng(), w3 = eng();
    std::printf("%u %u %u %u\n", w0, w1, w2, w3);
  }
  return 0;
}
