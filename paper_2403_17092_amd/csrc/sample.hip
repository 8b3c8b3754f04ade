// Layer-wise neighbour sampling and block construction.
//
// Per hop h (Neighbor Sampling, paper section 2.2; budgets of section 5.1.2),
// four kernels, none of which needs a count on the host:
//   1. sample:     one wavefront per dst node; Floyd's algorithm over CSR
//                  positions driven by Philox4x64-10 keyed by (rng_key, hop,
//                  node); the picks are ranked across the wave and the
//                  neighbours written, in ascending position order, into a
//                  padded [n_dst x fanout] layout (unused slots hold -1), so
//                  sampling does not wait for a prefix sum.  Each block also
//                  histograms the hash partitions of its keys in LDS.
//   2. partition:  scatter (key, padded position) pairs into hash partitions.
//   3. table:      one workgroup per partition builds an LDS open-addressing
//                  table recording, per key, the minimum position (atomicMin)
//                  and the number of occurrences; every element learns the
//                  first position of its key.  Padded positions preserve the
//                  (dst, position) order, so "first" is first occurrence.
//   4. scans:      one launch, two single-pass scans: the per-node counts into
//                  indptr, and the "position == first position" flags into
//                  local ids (first occurrences write src_nodes and src_occ).
// After the last hop one kernel compacts every hop's padded edges into the
// CSR indices (indices[e] = local id of the first occurrence of the key).
// The result does not depend on thread scheduling.
#include "internal.hpp"
#include "philox.hpp"
#include "sampler.hpp"
#include "wave.hpp"

namespace gnn {

namespace {

constexpr int kThreads = 256;
constexpr int kTableSlots = 4096;        // LDS table entries per partition
constexpr int kTargetPerPart = 2048;     // average elements per partition (upper bound)
constexpr int kMaxParts = 4096;
constexpr int32_t kEmpty = -1;
constexpr int kSampleThreads = 512;      // 8 waves per sampling block
constexpr int kSampleMaxBlocks = 1024;

// single-pass scan tiles
constexpr int kScanItems = 8;
constexpr int kScanTile = kThreads * kScanItems;

inline int partitions_for(int64_t cap_total) {
  int64_t want = ceil_div(cap_total > 0 ? cap_total : 1, kTargetPerPart);
  int p = 1;
  while (p < want && p < kMaxParts) p <<= 1;
  return p;
}

inline int log2i(int p) {
  int l = 0;
  while ((1 << l) < p) ++l;
  return l;
}

__device__ __forceinline__ uint32_t part_of(int32_t key, int log_parts) {
  uint32_t h = (uint32_t)key * 0x9E3779B1u;
  return log_parts ? (h >> (32 - log_parts)) : 0u;
}

__device__ __forceinline__ uint32_t slot_hash(int32_t key) {
  uint32_t h = (uint32_t)key * 0xCC9E2D51u;
  h ^= h >> 15;
  h *= 0x1B873593u;
  return h ^ (h >> 13);
}

// ---------------------------------------------------------------------------
// Single-pass exclusive scan (decoupled look-back, Merrill & Garland 2016).
// Tiles are taken in arrival order from a ticket counter, so a tile only ever
// waits on tiles whose blocks are already running.  Status word per tile:
// flag in the high half (0 empty, 1 tile aggregate, 2 inclusive prefix).
// ---------------------------------------------------------------------------
struct ScanState {
  int32_t* ticket;
  uint64_t* status;
};

__device__ __forceinline__ uint64_t scan_word(uint32_t flag, int32_t v) {
  return ((uint64_t)flag << 32) | (uint32_t)v;
}

__device__ __forceinline__ int32_t block_scan_excl(int32_t x, int32_t* total, int32_t* wsum) {
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const int32_t inc = wave_inclusive_scan(x);
  if (lane == 63) wsum[wid] = inc;
  __syncthreads();
  int32_t off = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < kThreads / 64; ++w) {
    off += (w < wid) ? wsum[w] : 0;
    tot += wsum[w];
  }
  __syncthreads();
  *total = tot;
  return off + inc - x;
}

// Scans load(i) for i < n; calls store(i, exclusive prefix, item) for i < n and
// finish(total) once (by the last tile).  Block-uniform early exit past n.
template <typename Load, typename Store, typename Finish>
__device__ __forceinline__ void tile_scan(ScanState ss, int64_t n, Load load, Store store, Finish finish) {
  __shared__ int32_t s_tile, s_prefix;
  __shared__ int32_t wsum[kThreads / 64];
  if (threadIdx.x == 0) s_tile = atomicAdd(ss.ticket, 1);
  __syncthreads();
  const int64_t tile = s_tile;
  int64_t ntiles = (n + kScanTile - 1) / kScanTile;
  ntiles = ntiles < 1 ? 1 : ntiles;
  if (tile >= ntiles) return;
  const int64_t base = tile * kScanTile + (int64_t)threadIdx.x * kScanItems;
  int32_t v[kScanItems];
  int32_t s = 0;
#pragma unroll
  for (int i = 0; i < kScanItems; ++i) {
    v[i] = (base + i < n) ? load(base + i) : 0;
    s += v[i];
  }
  int32_t agg;
  const int32_t excl = block_scan_excl(s, &agg, wsum);
  if (threadIdx.x == 0) {
    int32_t prefix = 0;
    if (tile == 0) {
      __hip_atomic_store(&ss.status[0], scan_word(2, agg), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    } else {
      __hip_atomic_store(&ss.status[tile], scan_word(1, agg), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      int64_t j = tile - 1;
      while (true) {
        const uint64_t w = __hip_atomic_load(&ss.status[j], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        const uint32_t f = (uint32_t)(w >> 32);
        if (f == 0) continue;
        prefix += (int32_t)(uint32_t)w;
        if (f == 2) break;
        --j;
      }
      __hip_atomic_store(&ss.status[tile], scan_word(2, prefix + agg), __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
    }
    s_prefix = prefix;
    if (tile == ntiles - 1) finish(prefix + agg);
  }
  __syncthreads();
  int32_t run = s_prefix + excl;
#pragma unroll
  for (int i = 0; i < kScanItems; ++i) {
    if (base + i < n) store(base + i, run, v[i]);
    run += v[i];
  }
}

inline int64_t scan_tiles(int64_t cap) { return std::max<int64_t>(1, ceil_div(cap, kScanTile)); }

// ---------------------------------------------------------------------------
// 1. sample (+ partition histogram): one wavefront per dst node, padded output
// ---------------------------------------------------------------------------
// Histogram copies spread the per-block flushes over more addresses.
inline int hist_copies(int parts) {
  int c = 8192 / parts;
  return c < 1 ? 1 : (c > 16 ? 16 : c);
}

template <typename RP>
__global__ void __launch_bounds__(kSampleThreads)
sample_kernel(const RP* __restrict__ rowptr, const int32_t* __restrict__ col, int64_t num_nodes,
              const int32_t* __restrict__ dst, const int32_t* n_src_dev, int32_t cap_dst,
              int32_t* counts, int32_t fanout, uint64_t rng_key, uint32_t hop,
              int32_t* __restrict__ nbr_pad, int32_t* __restrict__ kcount, int log_parts,
              int copies, int32_t* __restrict__ hist, int* err) {
  __shared__ int32_t lh[kMaxParts];
  const int parts = 1 << log_parts;
  for (int p = threadIdx.x; p < parts; p += kSampleThreads) lh[p] = 0;
  __syncthreads();
  const int lane = lane_id();
  int32_t n_dst = *n_src_dev;
  n_dst = n_dst > cap_dst ? cap_dst : n_dst;
  if (blockIdx.x == 0 && threadIdx.x == 0) counts[0] = n_dst;
  const int64_t waves = (int64_t)gridDim.x * (kSampleThreads / 64);
  for (int64_t i = ((int64_t)blockIdx.x * kSampleThreads + threadIdx.x) >> 6; i < n_dst; i += waves) {
    const int32_t v = dst[i];
    int32_t* out = nbr_pad + i * (int64_t)fanout;
    if (lane == 0) atomicAdd(&lh[part_of(v, log_parts)], 1);
    int32_t k = 0, w = -1;
    if (v < 0 || (int64_t)v >= num_nodes) {
      if (lane == 0) set_device_error(err, GNN_DEVERR_SEED_RANGE);
    } else {
      k = wave_sample(rowptr, col, v, fanout, rng_key, hop, &w);
    }
    if (lane == 0) kcount[i] = k;
    if (lane < fanout) out[lane] = w;
    if (lane < k) atomicAdd(&lh[part_of(w, log_parts)], 1);
  }
  __syncthreads();
  int32_t* hc = hist + (int64_t)(blockIdx.x % copies) * parts;
  for (int p = threadIdx.x; p < parts; p += kSampleThreads)
    if (lh[p]) atomicAdd(&hc[p], lh[p]);
}

// ---------------------------------------------------------------------------
// 3. partition: every block derives the partition offsets from the histogram,
//    reserves its slots per partition and writes (key, position) pairs.
// ---------------------------------------------------------------------------
// Key of padded position pos: the dst list, then the padded edge slots.
__device__ __forceinline__ int32_t key_at(int64_t pos, int32_t n_dst, const int32_t* dst,
                                          const int32_t* nbr_pad) {
  return pos < n_dst ? dst[pos] : nbr_pad[pos - n_dst];
}

__global__ void __launch_bounds__(kThreads)
partition_kernel(const int32_t* __restrict__ dst, const int32_t* __restrict__ nbr_pad,
                 const int32_t* counts, int32_t fanout, int log_parts, int copies,
                 const int32_t* __restrict__ hist, int32_t* __restrict__ part_start,
                 int32_t* __restrict__ cursor, int32_t* __restrict__ buf_key,
                 int32_t* __restrict__ buf_pos) {
  __shared__ int32_t lstart[kMaxParts];
  __shared__ int32_t lcount[kMaxParts];
  __shared__ int32_t wsum[kThreads / 64];
  const int parts = 1 << log_parts;
  const int32_t n_dst = counts[0];
  const int64_t total = (int64_t)n_dst * (1 + fanout);
  const int64_t base = (int64_t)blockIdx.x * kScanTile;
  if (base >= total && blockIdx.x != 0) return;
  // sum the histogram copies (coalesced reads, LDS atomics), then an exclusive
  // scan over the partitions (16 bins per thread) gives the offsets
  for (int p = threadIdx.x; p < parts; p += kThreads) lcount[p] = 0;
  __syncthreads();
  for (int idx = threadIdx.x; idx < parts * copies; idx += kThreads) {
    const int32_t x = hist[idx];
    if (x) atomicAdd(&lcount[idx & (parts - 1)], x);
  }
  __syncthreads();
  constexpr int kPer = kMaxParts / kThreads;
  int32_t hv[kPer];
  int32_t s = 0;
#pragma unroll
  for (int i = 0; i < kPer; ++i) {
    const int p = threadIdx.x * kPer + i;
    hv[i] = p < parts ? lcount[p] : 0;
    s += hv[i];
  }
  int32_t tot;
  int32_t off = block_scan_excl(s, &tot, wsum);
#pragma unroll
  for (int i = 0; i < kPer; ++i) {
    const int p = threadIdx.x * kPer + i;
    if (p < parts) {
      lstart[p] = off;
      lcount[p] = 0;
      if (blockIdx.x == 0) part_start[p] = off;
    }
    off += hv[i];
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) part_start[parts] = tot;
  __syncthreads();
  if (base >= total) return;
  int32_t keys[kScanItems];
  int32_t rank[kScanItems];
#pragma unroll
  for (int it = 0; it < kScanItems; ++it) {
    const int64_t pos = base + (int64_t)it * kThreads + threadIdx.x;
    keys[it] = pos < total ? key_at(pos, n_dst, dst, nbr_pad) : -1;
    rank[it] = keys[it] >= 0 ? atomicAdd(&lcount[part_of(keys[it], log_parts)], 1) : 0;
  }
  __syncthreads();
  for (int p = threadIdx.x; p < parts; p += kThreads)
    if (lcount[p]) lstart[p] += atomicAdd(&cursor[p], lcount[p]);
  __syncthreads();
#pragma unroll
  for (int it = 0; it < kScanItems; ++it) {
    const int64_t pos = base + (int64_t)it * kThreads + threadIdx.x;
    if (keys[it] >= 0) {
      const int32_t slot = lstart[part_of(keys[it], log_parts)] + rank[it];
      buf_key[slot] = keys[it];
      buf_pos[slot] = (int32_t)pos;
    }
  }
}

// ---------------------------------------------------------------------------
// 4. table
// ---------------------------------------------------------------------------
// Open-addressing insert / lookup on a table of `cap` slots.
__device__ __forceinline__ bool table_insert(int32_t* tk, int32_t* tm, int32_t* tc, uint32_t cap,
                                             int32_t key, int32_t pos) {
  uint32_t slot = slot_hash(key) % cap;
  for (uint32_t probe = 0; probe < cap; ++probe) {
    const int32_t old = atomicCAS(&tk[slot], kEmpty, key);
    if (old == kEmpty || old == key) {
      atomicMin(&tm[slot], pos);
      atomicAdd(&tc[slot], 1);
      return true;
    }
    slot = (slot + 1 == cap) ? 0 : slot + 1;
  }
  return false;
}

__device__ __forceinline__ uint32_t table_find(const int32_t* tk, uint32_t cap, int32_t key) {
  uint32_t slot = slot_hash(key) % cap;
  for (uint32_t probe = 0; probe < cap; ++probe) {
    if (tk[slot] == key) return slot;
    slot = (slot + 1 == cap) ? 0 : slot + 1;
  }
  return 0;  // unreachable: every looked-up key was inserted
}

__global__ void __launch_bounds__(kThreads)
table_kernel(const int32_t* __restrict__ part_start, const int32_t* __restrict__ buf_key,
             const int32_t* __restrict__ buf_pos, int32_t* __restrict__ first,
             int32_t* __restrict__ flag, int32_t* __restrict__ occ, int32_t* gkey, int32_t* gmin,
             int32_t* gcnt) {
  __shared__ int32_t tk[kTableSlots];
  __shared__ int32_t tm[kTableSlots];
  __shared__ int32_t tc[kTableSlots];
  __shared__ int overflow;
  const int p = blockIdx.x;
  const int32_t lo = part_start[p], hi = part_start[p + 1];
  if (lo >= hi) return;
  for (int s = threadIdx.x; s < kTableSlots; s += kThreads) {
    tk[s] = kEmpty;
    tm[s] = 0x7FFFFFFF;
    tc[s] = 0;
  }
  if (threadIdx.x == 0) overflow = 0;
  __syncthreads();
  bool ok = true;
  for (int32_t i = lo + threadIdx.x; i < hi; i += kThreads)
    ok &= table_insert(tk, tm, tc, kTableSlots, buf_key[i], buf_pos[i]);
  if (!ok) overflow = 1;
  __syncthreads();
  int32_t *K = tk, *Mn = tm, *Cn = tc;
  uint32_t cap = kTableSlots;
  if (overflow) {
    // more distinct keys than LDS slots: use this partition's global region
    cap = 2u * (uint32_t)(hi - lo);
    K = gkey + 2 * (int64_t)lo;
    Mn = gmin + 2 * (int64_t)lo;
    Cn = gcnt + 2 * (int64_t)lo;
    for (uint32_t s = threadIdx.x; s < cap; s += kThreads) {
      K[s] = kEmpty;
      Mn[s] = 0x7FFFFFFF;
      Cn[s] = 0;
    }
    __threadfence_block();
    __syncthreads();
    for (int32_t i = lo + threadIdx.x; i < hi; i += kThreads)
      table_insert(K, Mn, Cn, cap, buf_key[i], buf_pos[i]);
    __threadfence_block();
    __syncthreads();
  }
  for (int32_t i = lo + threadIdx.x; i < hi; i += kThreads) {
    const int32_t key = buf_key[i], pos = buf_pos[i];
    const uint32_t s = table_find(K, cap, key);
    const int32_t fp = Mn[s];
    first[pos] = fp;
    const bool is_first = (fp == pos);
    flag[pos] = is_first ? 1 : 0;
    if (is_first) occ[pos] = Cn[s];
  }
}

// ---------------------------------------------------------------------------
// 4. scans: blocks [0, count_blocks) scan the per-node counts into indptr
//    (counts[2] = E); the others scan the first-occurrence flags into local
//    ids (counts[1] = n_src) and emit src_nodes / src_occ.
// ---------------------------------------------------------------------------
__global__ void __launch_bounds__(kThreads)
scans_kernel(const int32_t* __restrict__ dst, const int32_t* __restrict__ nbr_pad, int32_t* counts,
             int32_t fanout, const int32_t* __restrict__ kcount, int32_t* __restrict__ indptr,
             int32_t count_blocks, const int32_t* __restrict__ flag, const int32_t* __restrict__ occ,
             int32_t* __restrict__ newid, int32_t cap_src, int32_t* __restrict__ src_nodes,
             int32_t* __restrict__ src_occ, ScanState s_cnt, ScanState s_flag, int* err) {
  const int32_t n_dst = counts[0];
  if ((int32_t)blockIdx.x < count_blocks) {
    auto load = [&](int64_t i) -> int32_t { return kcount[i]; };
    auto store = [&](int64_t i, int32_t pre, int32_t) { indptr[i] = pre; };
    auto finish = [&](int32_t total) {
      indptr[n_dst] = total;
      counts[2] = total;
    };
    tile_scan(s_cnt, n_dst, load, store, finish);
    return;
  }
  const int64_t n = (int64_t)n_dst * (1 + fanout);
  auto load = [&](int64_t i) -> int32_t {
    return (i < n_dst || nbr_pad[i - n_dst] >= 0) ? flag[i] : 0;
  };
  auto store = [&](int64_t i, int32_t id, int32_t f) {
    newid[i] = id;
    if (f) {
      if (id < cap_src) {
        src_nodes[id] = key_at(i, n_dst, dst, nbr_pad);
        src_occ[id] = occ[i];
      } else {
        set_device_error(err, GNN_DEVERR_CAPACITY);
      }
    }
  };
  auto finish = [&](int32_t total) { counts[1] = total; };
  tile_scan(s_flag, n, load, store, finish);
}

// ---------------------------------------------------------------------------
// finalize: compact padded slot (i, p), p < k_i, of every hop into
// indices[indptr[i] + p] = newid[first[n_dst + i * fanout + p]]
// ---------------------------------------------------------------------------
struct HopIndexArgs {
  int32_t* indices[GNN_MAX_LAYERS];
  const int32_t* indptr[GNN_MAX_LAYERS];
  const int32_t* kcount[GNN_MAX_LAYERS];
  const int32_t* first[GNN_MAX_LAYERS];
  const int32_t* newid[GNN_MAX_LAYERS];
  const int32_t* counts[GNN_MAX_LAYERS];
  int32_t fanout[GNN_MAX_LAYERS];
};

__global__ void __launch_bounds__(kThreads) indices_kernel(HopIndexArgs a) {
  const int h = blockIdx.y;
  const int32_t n_dst = a.counts[h][0];
  const int32_t f = a.fanout[h];
  const int64_t slots = (int64_t)n_dst * f;
  for (int64_t s = (int64_t)blockIdx.x * kThreads + threadIdx.x; s < slots;
       s += (int64_t)gridDim.x * kThreads) {
    const int64_t i = s / f;
    const int32_t p = (int32_t)(s - i * f);
    if (p < a.kcount[h][i]) a.indices[h][a.indptr[h][i] + p] = a.newid[h][a.first[h][n_dst + s]];
  }
}

}  // namespace

// Scratch layout of one gnn_sample_blocks call.  Padded position space of hop
// h: n_dst + n_dst * fanout (<= cap_dst[h] * (1 + fanout) = cap_total).
struct SampleScratch {
  int32_t* hist[GNN_MAX_LAYERS];        // [copies x kMaxParts]
  int32_t* cursor[GNN_MAX_LAYERS];      // [kMaxParts]
  int32_t* part_start[GNN_MAX_LAYERS];  // [kMaxParts + 1]
  int32_t* kcount[GNN_MAX_LAYERS];      // [cap_dst]
  int32_t* first[GNN_MAX_LAYERS];       // [cap_total]
  int32_t* newid[GNN_MAX_LAYERS];       // [cap_total]
  int32_t* tickets;                     // [2 L]
  uint64_t* status[2 * GNN_MAX_LAYERS]; // scan tile status
  int32_t* buf_key;                     // [max_total]
  int32_t* buf_pos;
  int32_t* flag;
  int32_t* occ;
  int32_t* gkey;                        // [2 max_total] fallback tables
  int32_t* gmin;
  int32_t* gcnt;
  void* zero_begin;                     // [zero_begin, zero_end): cleared once per call
  void* zero_end;
};

static size_t carve_sample(Carver& c, const int32_t* cap_dst, const int64_t* cap_edges, int32_t L,
                           SampleScratch* s) {
  int64_t max_total = 1;
  for (int h = 0; h < L; ++h) max_total = std::max<int64_t>(max_total, (int64_t)cap_dst[h] + cap_edges[h]);
  // the region cleared at the start of every call comes first
  s->zero_begin = c.take<char>(0);
  for (int h = 0; h < L; ++h) {
    s->hist[h] = c.take<int32_t>(16 * kMaxParts);
    s->cursor[h] = c.take<int32_t>(kMaxParts);
  }
  s->tickets = c.take<int32_t>(2 * GNN_MAX_LAYERS);
  for (int h = 0; h < L; ++h) {
    s->status[2 * h] = c.take<uint64_t>(scan_tiles(cap_dst[h]));
    s->status[2 * h + 1] = c.take<uint64_t>(scan_tiles((int64_t)cap_dst[h] + cap_edges[h]));
  }
  s->zero_end = c.take<char>(0);
  for (int h = 0; h < L; ++h) {
    const int64_t tot = (int64_t)cap_dst[h] + cap_edges[h];
    s->part_start[h] = c.take<int32_t>(kMaxParts + 1);
    s->kcount[h] = c.take<int32_t>(std::max<int64_t>(1, cap_dst[h]));
    s->first[h] = c.take<int32_t>(std::max<int64_t>(1, tot));
    s->newid[h] = c.take<int32_t>(std::max<int64_t>(1, tot));
  }
  s->buf_key = c.take<int32_t>(max_total);
  s->buf_pos = c.take<int32_t>(max_total);
  s->flag = c.take<int32_t>(max_total);
  s->occ = c.take<int32_t>(max_total);
  s->gkey = c.take<int32_t>(2 * max_total);
  s->gmin = c.take<int32_t>(2 * max_total);
  s->gcnt = c.take<int32_t>(2 * max_total);
  return c.off;
}

size_t sample_scratch_bytes(const int32_t* cap_dst, const int32_t* cap_src,
                            const int64_t* cap_edges, int32_t L) {
  (void)cap_src;
  Carver c(nullptr, 0);
  SampleScratch s;
  return carve_sample(c, cap_dst, cap_edges, L, &s);
}

template <typename RP>
static int sample_hops(const gnn_csr* csr, const RP* rowptr, const int32_t* seeds, int32_t B,
                       const int32_t* fanouts, int32_t L, uint64_t rng_key, gnn_block* blocks,
                       void* ws, size_t ws_bytes, hipStream_t st) {
  int32_t cap_dst[GNN_MAX_LAYERS];
  int64_t cap_edges[GNN_MAX_LAYERS];
  for (int h = 0; h < L; ++h) {
    cap_dst[h] = blocks[h].cap_dst;
    cap_edges[h] = blocks[h].cap_edges;
    if (cap_edges[h] != (int64_t)cap_dst[h] * fanouts[h])
      return fail(GNN_EINVAL, "gnn_sample_blocks: cap_edges must equal cap_dst * fanout");
  }
  Carver c(ws, ws_bytes);
  SampleScratch sc;
  carve_sample(c, cap_dst, cap_edges, L, &sc);
  if (!c.fits()) return fail(GNN_EWORKSPACE, "gnn_sample_blocks: workspace %zu < %zu bytes", ws_bytes, c.off);
  int* err = device_error_word();
  if (!err) return fail(GNN_EHIP, "device error word unavailable");

  // hop 1's dst count lives in blocks[0].counts[0]; clear histograms, cursors
  // and scan state for every hop in one launch
  const int64_t zero_words =
      (static_cast<char*>(sc.zero_end) - static_cast<char*>(sc.zero_begin)) / 4;
  FillRange fr[2] = {{blocks[0].counts, 1, B}, {sc.zero_begin, zero_words, 0}};
  if (int rc = launch_fill(fr, 2, st)) return rc;

  HopIndexArgs ia{};
  int64_t max_slots = 1;
  for (int h = 0; h < L; ++h) {
    gnn_block& bk = blocks[h];
    const int32_t* dst = h == 0 ? seeds : blocks[h - 1].src_nodes;
    const int32_t* n_dst_src = h == 0 ? blocks[0].counts : blocks[h - 1].counts + 1;
    const int32_t f = fanouts[h];
    const int64_t cap_total = (int64_t)bk.cap_dst + bk.cap_edges;
    const int parts = partitions_for(cap_total);
    const int lp = log2i(parts);
    const int copies = hist_copies(parts);

    const int64_t sblocks = std::min<int64_t>(kSampleMaxBlocks,
                                              std::max<int64_t>(1, ceil_div(bk.cap_dst, kSampleThreads / 64)));
    sample_kernel<RP><<<(unsigned)sblocks, kSampleThreads, 0, st>>>(
        rowptr, csr->col, csr->num_nodes, dst, n_dst_src, bk.cap_dst, bk.counts, f, rng_key,
        (uint32_t)(h + 1), bk.indices, sc.kcount[h], lp, copies, sc.hist[h], err);
    partition_kernel<<<(unsigned)scan_tiles(cap_total), kThreads, 0, st>>>(
        dst, bk.indices, bk.counts, f, lp, copies, sc.hist[h], sc.part_start[h], sc.cursor[h],
        sc.buf_key, sc.buf_pos);
    table_kernel<<<parts, kThreads, 0, st>>>(sc.part_start[h], sc.buf_key, sc.buf_pos, sc.first[h],
                                             sc.flag, sc.occ, sc.gkey, sc.gmin, sc.gcnt);
    ScanState s_cnt{sc.tickets + 2 * h, sc.status[2 * h]};
    ScanState s_flag{sc.tickets + 2 * h + 1, sc.status[2 * h + 1]};
    const int64_t cb = scan_tiles(bk.cap_dst), fb = scan_tiles(cap_total);
    scans_kernel<<<(unsigned)(cb + fb), kThreads, 0, st>>>(
        dst, bk.indices, bk.counts, f, sc.kcount[h], bk.indptr, (int32_t)cb, sc.flag, sc.occ,
        sc.newid[h], bk.cap_src, bk.src_nodes, bk.src_occ, s_cnt, s_flag, err);
    GNN_LAUNCH_CHECK("gnn_sample_blocks");
    ia.indices[h] = bk.indices;
    ia.indptr[h] = bk.indptr;
    ia.kcount[h] = sc.kcount[h];
    ia.first[h] = sc.first[h];
    ia.newid[h] = sc.newid[h];
    ia.counts[h] = bk.counts;
    ia.fanout[h] = f;
    max_slots = std::max<int64_t>(max_slots, bk.cap_edges);
  }
  const int64_t gx = std::min<int64_t>(2048, std::max<int64_t>(1, ceil_div(max_slots, kThreads * 4)));
  indices_kernel<<<dim3((unsigned)gx, (unsigned)L), kThreads, 0, st>>>(ia);
  GNN_LAUNCH_CHECK("gnn_sample_blocks indices");
  return GNN_OK;
}

int sample_blocks_impl(const gnn_csr* csr, const int32_t* seeds, int32_t B, const int32_t* fanouts,
                       int32_t L, uint64_t rng_key, gnn_block* blocks, void* ws, size_t ws_bytes,
                       hipStream_t st) {
  if (csr->rowptr_bits == 64)
    return sample_hops(csr, static_cast<const int64_t*>(csr->rowptr), seeds, B, fanouts, L, rng_key,
                       blocks, ws, ws_bytes, st);
  return sample_hops(csr, static_cast<const int32_t*>(csr->rowptr), seeds, B, fanouts, L, rng_key,
                     blocks, ws, ws_bytes, st);
}

}  // namespace gnn

// ---------------------------------------------------------------------------
// C ABI
// ---------------------------------------------------------------------------
extern "C" {

int gnn_block_caps(int32_t B, const int32_t* fanouts, int32_t L, int64_t N, int32_t* cap_dst,
                   int32_t* cap_src, int64_t* cap_edges) {
  using namespace gnn;
  if (!fanouts || !cap_dst || !cap_src || !cap_edges) return fail(GNN_EINVAL, "gnn_block_caps: null pointer");
  if (L < 1 || L > GNN_MAX_LAYERS) return fail(GNN_EINVAL, "gnn_block_caps: L=%d not in [1, %d]", L, GNN_MAX_LAYERS);
  if (B < 0 || N < 0) return fail(GNN_EINVAL, "gnn_block_caps: negative size");
  int64_t nd = B;
  for (int h = 0; h < L; ++h) {
    if (fanouts[h] < 1 || fanouts[h] > GNN_MAX_FANOUT)
      return fail(GNN_EINVAL, "gnn_block_caps: fanout %d not in [1, %d]", fanouts[h], GNN_MAX_FANOUT);
    const int64_t e = nd * fanouts[h];
    int64_t ns = nd + e;
    if (ns > N && N >= nd) ns = N;
    if (e > INT32_MAX || ns > INT32_MAX) return fail(GNN_EINVAL, "gnn_block_caps: block too large");
    cap_dst[h] = (int32_t)nd;
    cap_edges[h] = e;
    cap_src[h] = (int32_t)ns;
    nd = ns;
  }
  return GNN_OK;
}

size_t gnn_sample_workspace_bytes(int32_t B, const int32_t* fanouts, int32_t L, int64_t N) {
  int32_t cd[GNN_MAX_LAYERS], cs[GNN_MAX_LAYERS];
  int64_t ce[GNN_MAX_LAYERS];
  if (gnn_block_caps(B, fanouts, L, N, cd, cs, ce) != GNN_OK) return 0;
  return gnn::sample_scratch_bytes(cd, cs, ce, L);
}

int gnn_sample_blocks(const gnn_csr* csr, const int32_t* seeds, int32_t B, const int32_t* fanouts,
                      int32_t L, uint64_t rng_key, gnn_block* blocks, void* ws, size_t ws_bytes,
                      void* stream) {
  using namespace gnn;
  if (!csr || !blocks || !fanouts || !ws) return fail(GNN_EINVAL, "gnn_sample_blocks: null pointer");
  if (!csr->rowptr || !csr->col) return fail(GNN_EINVAL, "gnn_sample_blocks: null CSR array");
  if (csr->rowptr_bits != 32 && csr->rowptr_bits != 64)
    return fail(GNN_EINVAL, "gnn_sample_blocks: rowptr_bits must be 32 or 64");
  if (csr->num_nodes < 0 || csr->num_nodes > INT32_MAX)
    return fail(GNN_EINVAL, "gnn_sample_blocks: num_nodes out of range");
  if (B < 0 || (B > 0 && !seeds)) return fail(GNN_EINVAL, "gnn_sample_blocks: bad seeds");
  int32_t cd[GNN_MAX_LAYERS], cs[GNN_MAX_LAYERS];
  int64_t ce[GNN_MAX_LAYERS];
  if (int rc = gnn_block_caps(B, fanouts, L, csr->num_nodes, cd, cs, ce)) return rc;
  for (int h = 0; h < L; ++h) {
    const gnn_block& b = blocks[h];
    if (!b.indptr || !b.indices || !b.src_nodes || !b.src_occ || !b.counts)
      return fail(GNN_EINVAL, "gnn_sample_blocks: block %d has a null array", h);
    if (b.cap_dst < cd[h] || b.cap_src < cs[h] || b.cap_edges < ce[h])
      return fail(GNN_EWORKSPACE, "gnn_sample_blocks: block %d capacities below gnn_block_caps", h);
  }
  // the dst list of hop h+1 is the src list of hop h: its capacity must match
  for (int h = 1; h < L; ++h)
    if (blocks[h].cap_dst < blocks[h - 1].cap_src)
      return fail(GNN_EWORKSPACE, "gnn_sample_blocks: block %d cap_dst < block %d cap_src", h, h - 1);
  if (ws_bytes < sample_scratch_bytes(cd, cs, ce, L))
    return fail(GNN_EWORKSPACE, "gnn_sample_blocks: workspace too small");
  // the kernels size their grids from the capacities given in `blocks`
  gnn_block local[GNN_MAX_LAYERS];
  for (int h = 0; h < L; ++h) {
    local[h] = blocks[h];
    local[h].cap_dst = cd[h];
    local[h].cap_src = blocks[h].cap_src;
    local[h].cap_edges = ce[h];
  }
  return sample_blocks_impl(csr, seeds, B, fanouts, L, rng_key, local, ws, ws_bytes, as_stream(stream));
}

}  // extern "C"
