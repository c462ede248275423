// Counter-based random draws for temperature sampling: Philox-4x32 with 10
// rounds (Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as easy as
// 1, 2, 3", SC 2011).  A draw is a pure function of (seed, stream, batch row,
// depth, vocabulary id): counter = (v / 4, depth, row, stream), key = the
// 64-bit seed, word v % 4 of the block.  A word x maps to the uniform
// (floor(x / 2^9) + 1/2) / 2^23, exactly representable in fp32, in (0, 1).
#pragma once
#include "common.h"

namespace dk {

enum { RNG_DRAFT = 0, RNG_ACCEPT = 1, RNG_BONUS = 2 };

struct Philox4 {
  uint32_t x[4];
};

DEVI Philox4 philox4x32_10(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3, uint32_t k0, uint32_t k1) {
  constexpr uint32_t kM0 = 0xD2511F53u, kM1 = 0xCD9E8D57u, kW0 = 0x9E3779B9u, kW1 = 0xBB67AE85u;
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    const uint32_t hi0 = __umulhi(kM0, c0), lo0 = kM0 * c0;
    const uint32_t hi1 = __umulhi(kM1, c2), lo1 = kM1 * c2;
    const uint32_t n0 = hi1 ^ c1 ^ k0, n2 = hi0 ^ c3 ^ k1;
    c0 = n0;
    c1 = lo1;
    c2 = n2;
    c3 = lo0;
    k0 += kW0;
    k1 += kW1;
  }
  return Philox4{{c0, c1, c2, c3}};
}

DEVI float rng_uniform(uint32_t x) { return ((float)(x >> 9) + 0.5f) * (1.0f / 8388608.0f); }
DEVI float rng_gumbel(uint32_t x) { return -logf(-logf(rng_uniform(x))); }

// The four words of vocabulary ids 4*v4 .. 4*v4+3 for (seed, stream, row, depth).
DEVI Philox4 rng_block(uint32_t seed_lo, uint32_t seed_hi, int stream, int row, int depth, int v4) {
  return philox4x32_10((uint32_t)v4, (uint32_t)depth, (uint32_t)row, (uint32_t)stream, seed_lo, seed_hi);
}

}  // namespace dk
