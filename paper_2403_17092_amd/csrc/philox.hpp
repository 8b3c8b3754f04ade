// Philox4x64-10 on the GPU (Salmon, Moraes, Dror, Shaw, "Parallel Random
// Numbers: As Easy as 1, 2, 3", SC'11): ten rounds of two 64x64->128-bit
// multiplies, key bumped by two Weyl increments between rounds.
#pragma once
#include <hip/hip_runtime.h>

#include <cstdint>

namespace gnn {

struct U64x4 {
  uint64_t x[4];
};

__device__ __forceinline__ U64x4 philox4x64_10(uint64_t c0, uint64_t c1, uint64_t c2, uint64_t c3,
                                               uint64_t k0, uint64_t k1) {
  constexpr uint64_t kM0 = 0xD2E7470EE14C6C93ull;
  constexpr uint64_t kM1 = 0xCA5A826395121157ull;
  constexpr uint64_t kW0 = 0x9E3779B97F4A7C15ull;
  constexpr uint64_t kW1 = 0xBB67AE8584CAA73Bull;
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r) {
      k0 += kW0;
      k1 += kW1;
    }
    const uint64_t hi0 = __umul64hi(kM0, c0), lo0 = kM0 * c0;
    const uint64_t hi1 = __umul64hi(kM1, c2), lo1 = kM1 * c2;
    const uint64_t n0 = hi1 ^ c1 ^ k0;
    const uint64_t n2 = hi0 ^ c3 ^ k1;
    c0 = n0;
    c1 = lo1;
    c2 = n2;
    c3 = lo0;
  }
  return U64x4{{c0, c1, c2, c3}};
}

// Draw s of node v at hop h: word (s mod 4) of the block at counter
// (1 + s/4, v, h, 0) under key (rng_key, 0).
__device__ __forceinline__ uint64_t sample_draw(uint64_t rng_key, uint32_t hop, uint32_t node,
                                                uint32_t s) {
  U64x4 y = philox4x64_10(1ull + (s >> 2), node, hop, 0ull, rng_key, 0ull);
  const uint32_t w = s & 3u;
  return w == 0 ? y.x[0] : (w == 1 ? y.x[1] : (w == 2 ? y.x[2] : y.x[3]));
}

// floor(r * m / 2^64): a uniform integer in [0, m).
__device__ __forceinline__ uint32_t bounded_draw(uint64_t r, uint32_t m) {
  return (uint32_t)__umul64hi(r, (uint64_t)m);
}

}  // namespace gnn
