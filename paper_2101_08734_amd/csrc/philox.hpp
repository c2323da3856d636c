// Philox-4x32-10 on the device (Salmon, Moraes, Dror, Shaw, "Parallel Random
// Numbers: As Easy as 1, 2, 3", SC'11): a counter-based generator, so the key
// of any (epoch, sample) is computed directly from the seed without state.
//
// Shuffle keys: the keys of samples 4c .. 4c+3 in epoch e are the four output
// words of the block at counter (c, e, 0, 0) under key (seed lo, seed hi).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace nopfs {

struct Philox4 {
  uint32_t x, y, z, w;
};

// Round multipliers and the Weyl increments of the round key, as published.
constexpr uint32_t kPhiloxMulA = 0xD2511F53u;
constexpr uint32_t kPhiloxMulB = 0xCD9E8D57u;
constexpr uint32_t kPhiloxWeylA = 0x9E3779B9u;
constexpr uint32_t kPhiloxWeylB = 0xBB67AE85u;

// One block with words 2 and 3 of the counter equal to zero. The round key
// is uniform across lanes, so its schedule stays in scalar registers.
__device__ __forceinline__ Philox4 philox_block(uint32_t c0, uint32_t c1, uint32_t k0,
                                                uint32_t k1) {
  uint32_t a = c0, b = c1, c = 0u, d = 0u;
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    const uint64_t pa = uint64_t(kPhiloxMulA) * a;
    const uint64_t pc = uint64_t(kPhiloxMulB) * c;
    const uint32_t na = uint32_t(pc >> 32) ^ b ^ k0;
    const uint32_t nb = uint32_t(pc);
    const uint32_t nc = uint32_t(pa >> 32) ^ d ^ k1;
    const uint32_t nd = uint32_t(pa);
    a = na; b = nb; c = nc; d = nd;
    k0 += kPhiloxWeylA;
    k1 += kPhiloxWeylB;
  }
  return Philox4{a, b, c, d};
}

}  // namespace nopfs
