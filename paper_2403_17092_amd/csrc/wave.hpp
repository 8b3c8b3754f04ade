// Wave64 primitives for CDNA (gfx950).
#pragma once
#include <hip/hip_runtime.h>

#include <cstdint>

namespace gnn {

constexpr int WAVE = 64;

__device__ inline int lane_id() { return __lane_id(); }

// Inclusive prefix sum across the 64 lanes of a wave.
__device__ inline int32_t wave_inclusive_scan(int32_t x) {
  const int lane = lane_id();
#pragma unroll
  for (int d = 1; d < WAVE; d <<= 1) {
    int32_t y = __shfl_up(x, d, WAVE);
    if (lane >= d) x += y;
  }
  return x;
}

__device__ inline float wave_sum(float x) {
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) x += __shfl_xor(x, d, WAVE);
  return x;
}

__device__ inline float wave_max(float x) {
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) x = fmaxf(x, __shfl_xor(x, d, WAVE));
  return x;
}

__device__ inline uint64_t ballot(bool p) { return __ballot(p); }

// Uniform (wave-wide) read of lane `l`'s value; `l` must be wave-uniform.
__device__ inline int32_t read_lane(int32_t x, int l) { return __builtin_amdgcn_readlane(x, l); }

__device__ inline void set_device_error(int* word, int bit) {
  if (word) atomicOr(word, bit);
}

}  // namespace gnn
