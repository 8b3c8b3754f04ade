// Wave-level uniform neighbour sampling without replacement (shared by the
// layer-wise sampler and the ShaDow extractor).
#pragma once
#include "philox.hpp"
#include "wave.hpp"

namespace gnn {

template <typename RP>
__device__ __forceinline__ void row_range(const RP* rowptr, int32_t v, int64_t& start, int64_t& deg) {
  start = (int64_t)rowptr[v];
  deg = (int64_t)rowptr[v + 1] - start;
}

// The whole wave samples node v (valid id) at hop `hop`: k = min(fanout, d)
// neighbours.  On return, lane `rank` (rank < k) holds the rank-th chosen
// neighbour in ascending CSR position order in *nbr; the function returns k.
// If d <= fanout all neighbours are taken and no random number is drawn;
// otherwise Floyd's algorithm picks k distinct positions: step s draws t_s
// uniform in [0, j_s], j_s = d - k + s (draw s of Philox4x64-10 at counter
// (1 + s/4, v, hop, 0), key (rng_key, 0)), and keeps t_s unless an earlier
// step chose it, in which case it keeps j_s.  Must be called by all 64 lanes
// (fanout <= 64).
template <typename RP>
__device__ __forceinline__ int32_t wave_sample(const RP* __restrict__ rowptr,
                                               const int32_t* __restrict__ col, int32_t v,
                                               int32_t fanout, uint64_t rng_key, uint32_t hop,
                                               int32_t* nbr) {
  const int lane = lane_id();
  int64_t start, d;
  row_range(rowptr, v, start, d);
  if (d <= fanout) {
    *nbr = lane < d ? col[start + lane] : -1;
    return (int32_t)d;
  }
  const uint32_t du = (uint32_t)d;
  const uint32_t f = (uint32_t)fanout;
  uint32_t t = 0;
  if ((uint32_t)lane < f) {
    const uint64_t r = sample_draw(rng_key, hop, (uint32_t)v, (uint32_t)lane);
    t = bounded_draw(r, du - f + (uint32_t)lane + 1u);
  }
  int32_t pick = -1;
  for (uint32_t s = 0; s < f; ++s) {
    const int32_t ts = read_lane((int32_t)t, (int)s);
    const bool dup = ballot((uint32_t)lane < s && pick == ts) != 0ull;
    const int32_t chosen = dup ? (int32_t)(du - f + s) : ts;
    if ((uint32_t)lane == s) pick = chosen;
  }
  // rank of each pick among the f distinct picks -> ascending position order
  int32_t rank = 0;
  for (uint32_t m = 0; m < f; ++m) {
    const int32_t pm = read_lane(pick, (int)m);
    rank += (pm < pick) ? 1 : 0;
  }
  // move pick of rank r to lane r
  const int32_t w = (uint32_t)lane < f ? col[start + pick] : -1;
  int32_t src_lane = 0;
  for (uint32_t m = 0; m < f; ++m) {
    const int32_t rm = read_lane(rank, (int)m);
    if (rm == lane) src_lane = (int32_t)m;
  }
  const int32_t moved = __shfl(w, src_lane, 64);
  *nbr = (uint32_t)lane < f ? moved : -1;
  return (int32_t)f;
}

// The same sampling done by a group of G lanes (G = 16, 32 or 64, fanout <=
// G), so a wave samples 64 / G nodes at once: lanes [g0, g0 + G) with
// g0 = lane & ~(G - 1) sample node v of their group (valid == false: an empty
// row).  Lane g0 + r of the group holds the rank-r neighbour (-1 for r >= k)
// in *nbr; every lane of the group returns k.  fanout must be the same for the
// whole wave, and every lane of the wave must call it.
template <int G, typename RP>
__device__ __forceinline__ int32_t group_sample(const RP* __restrict__ rowptr,
                                                const int32_t* __restrict__ col, bool valid,
                                                int32_t v, int32_t fanout, uint64_t rng_key,
                                                uint32_t hop, int32_t* nbr) {
  static_assert(G == 16 || G == 32 || G == 64, "group size");
  // value of lane g0 + s of the group (a scalar read when the group is the wave)
  auto bcast = [](int32_t x, int g0, int s) -> int32_t {
    return G == 64 ? read_lane(x, s) : __shfl(x, g0 + s, WAVE);
  };
  const int lane = lane_id();
  const int r = lane & (G - 1);
  const int g0 = lane - r;
  const uint64_t gmask = G == 64 ? ~0ull : (((1ull << G) - 1ull) << g0);
  int64_t start = 0, d = 0;
  if (valid) row_range(rowptr, v, start, d);
  const bool all = d <= fanout;
  const uint32_t du = (uint32_t)d;
  const uint32_t f = (uint32_t)fanout;
  uint32_t t = 0;
  if (!all && (uint32_t)r < f) {
    const uint64_t x = sample_draw(rng_key, hop, (uint32_t)v, (uint32_t)r);
    t = bounded_draw(x, du - f + (uint32_t)r + 1u);
  }
  // Floyd: step s keeps t_s unless an earlier step of the group chose it
  int32_t pick = -1;
  for (uint32_t s = 0; s < f; ++s) {
    const int32_t ts = bcast((int32_t)t, g0, (int)s);
    const bool dup = (ballot((uint32_t)r < s && pick == ts) & gmask) != 0ull;
    const int32_t chosen = dup ? (int32_t)(du - f + s) : ts;
    if ((uint32_t)r == s) pick = chosen;
  }
  // rank of each pick among the group's f picks -> ascending position order;
  // then lane r fetches the pick of rank r
  int32_t rank = 0, src = 0;
  for (uint32_t m = 0; m < f; ++m) {
    const int32_t pm = bcast(pick, g0, (int)m);
    rank += (pm < pick) ? 1 : 0;
  }
  for (uint32_t m = 0; m < f; ++m) {
    const int32_t rm = bcast(rank, g0, (int)m);
    if (rm == r) src = (int32_t)m;
  }
  const int32_t pos = __shfl(pick, g0 + src, WAVE);
  if (all) {
    *nbr = r < d ? col[start + r] : -1;
    return (int32_t)d;
  }
  *nbr = (uint32_t)r < f ? col[start + pos] : -1;
  return (int32_t)f;
}

}  // namespace gnn
