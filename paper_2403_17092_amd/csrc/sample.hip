// Layer-wise neighbour sampling and block construction.
//
// Per hop h (Neighbor Sampling, paper section 2.2; budgets of section 5.1.2),
// two launches, none of which needs a count on the host:
//   1. sample:  a group of 16, 32 or 64 lanes (the smallest that holds the
//               fanout) per dst node; Floyd's algorithm over CSR
//               positions driven by Philox4x64-10 keyed by (rng_key, hop,
//               node); the picks are ranked across the wave and written, in
//               ascending position order, into a padded [n_dst x fanout]
//               layout (unused slots hold -1), so sampling does not wait for
//               a prefix sum.  The padded position space is the dst list
//               followed by the padded slots, i.e. (dst index, rank) order.
//               Every key records itself in a per-node word with a 64-bit
//               atomicMax of (epoch << 32 | ~position), so after the launch
//               the word of a node holds the first position at which it
//               occurs in this hop.  The same launch compacts the previous
//               hop's edges (step 3), which needs that hop's local ids.
//   2. scans:   two single-pass scans in one launch: the per-node counts
//               into indptr, and the first-occurrence flags into local ids;
//               each first occurrence writes src_nodes, the initial src_occ
//               (1 for dst nodes, else 0) and its node's local id into a
//               per-node table.
//   3. indices: padded slot (i, r), r < k_i, becomes indices[indptr[i] + r] =
//               the local id of its key, and adds 1 to src_occ of that id.
// The last hop's step 3 is a launch of its own.  Words of earlier hops and
// calls carry smaller epochs and lose every atomicMax, so the per-node arrays
// are cleared only when the workspace header says they were not built by an
// earlier call for this node count.  The result does not depend on thread
// scheduling.
#include <atomic>

#include "internal.hpp"
#include "philox.hpp"
#include "relabel.hpp"
#include "sampler.hpp"
#include "wave.hpp"

namespace gnn {

namespace {

constexpr int kThreads = 256;
constexpr int kSampleThreads = 512;      // 8 waves per sampling block
constexpr int kSampleMaxBlocks = 1024;
constexpr int kIndexBlocksMax = 1024;
constexpr int kBeginBlocks = 256;
constexpr int kMaxExtraFills = 4;
constexpr int64_t kResidentWaves = 8192;  // 256 CUs x 32 waves
// scan blocks (256 threads, 8 KB of LDS at most) that are certainly resident
// at once: 256 CUs x 4
constexpr int64_t kResidentScanBlocks = 1024;

// single-pass scan tiles
// single-pass scan tiles: ITEMS per thread, the smallest of 2, 4, 8 whose
// grid is resident at once (small tiles keep more blocks in flight)
constexpr int kScanItemsMin = 2;
constexpr int kScanItemsMax = 8;

// Per-node word of the first-occurrence race: epoch in the high half, the
// complemented position in the low half (so atomicMax keeps the newest epoch
// and, within it, the smallest position).
__device__ __forceinline__ uint64_t occ_word(uint32_t epoch, int64_t pos) {
  return ((uint64_t)epoch << 32) | (uint32_t)~(uint32_t)pos;
}

// ---------------------------------------------------------------------------
// Single-pass exclusive scan (decoupled look-back, Merrill & Garland 2016).
// Tiles are taken in arrival order from a ticket counter, so a tile only ever
// waits on tiles whose blocks are already running.  Status word per tile:
// flag in the high half (0 empty, 1 tile aggregate, 2 inclusive prefix).  The
// look-back reads 64 predecessors at once, one per lane of the first wave.
// ---------------------------------------------------------------------------
struct ScanState {
  int32_t* ticket;
  uint64_t* status;
  int* err;  // device error word (a look-back that gives up sets GNN_DEVERR_SYNC)
};

// Look-back reads of an unpublished predecessor before the wait gives up
// (far beyond any live wait: a predecessor that runs publishes within
// microseconds).  Giving up treats the unread predecessors as zero, so every
// prefix stays at or below the true one and every store stays in bounds.
constexpr int32_t kScanSpinLimit = 1 << 22;

__device__ __forceinline__ uint64_t scan_word(uint32_t flag, int32_t v) {
  return ((uint64_t)flag << 32) | (uint32_t)v;
}

__device__ __forceinline__ int32_t wave_sum_i32(int32_t x) {
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) x += __shfl_xor(x, d, WAVE);
  return x;
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

// Exclusive prefix of `tile` given its aggregate; run by the whole first wave.
__device__ __forceinline__ int32_t look_back(ScanState ss, int64_t tile, int32_t agg) {
  const int lane = threadIdx.x & 63;
  if (tile == 0) {
    if (lane == 0)
      __hip_atomic_store(&ss.status[0], scan_word(2, agg), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    return 0;
  }
  if (lane == 0)
    __hip_atomic_store(&ss.status[tile], scan_word(1, agg), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  int32_t prefix = 0;
  int64_t top = tile - 1;  // the window holds tiles top, top - 1, ..., top - 63
  int32_t spins = 0;
  while (true) {
    const int64_t j = top - lane;
    const uint64_t w = j >= 0 ? __hip_atomic_load(&ss.status[j], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)
                              : scan_word(2, 0);  // before tile 0: an inclusive 0
    const uint32_t f = (uint32_t)(w >> 32);
    const uint64_t incl = ballot(f == 2);
    const uint64_t empty = ballot(f == 0);
    const int stop = incl ? __builtin_ctzll(incl) : 64;       // nearest inclusive prefix
    const uint64_t need = stop >= 63 ? ~0ull : ((2ull << stop) - 1);
    if (empty & need) {  // a predecessor has not published yet
      if (++spins <= kScanSpinLimit) continue;
      // bounded wait: flag the error and go on with what has been published
      if (lane == 0) set_device_error(ss.err, GNN_DEVERR_SYNC);
      const bool take = lane <= stop && !((empty >> lane) & 1ull);
      prefix += wave_sum_i32(take ? (int32_t)(uint32_t)w : 0);
      break;
    }
    prefix += wave_sum_i32(lane <= stop ? (int32_t)(uint32_t)w : 0);
    if (stop < 64) break;
    top -= 64;
  }
  if (lane == 0)
    __hip_atomic_store(&ss.status[tile], scan_word(2, prefix + agg), __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
  return prefix;
}

// Scans load(i) for i < n; calls store(i, exclusive prefix, item) for i < n and
// finish(total) once (by the last tile).  Block-uniform early exit past n.
// tile_id < 0 takes the tile from the ticket counter (arrival order);
// otherwise the caller guarantees every lower tile's block runs concurrently.
template <int ITEMS, typename Load, typename Store, typename Finish>
__device__ __forceinline__ void tile_scan(ScanState ss, int64_t tile_id, int64_t n, Load load,
                                          Store store, Finish finish) {
  __shared__ int32_t s_tile, s_prefix;
  __shared__ int32_t wsum[kThreads / 64];
  if (tile_id < 0) {
    if (threadIdx.x == 0) s_tile = atomicAdd(ss.ticket, 1);
    __syncthreads();
    tile_id = s_tile;
  }
  const int64_t tile = tile_id;
  constexpr int kTile = kThreads * ITEMS;
  int64_t ntiles = (n + kTile - 1) / kTile;
  ntiles = ntiles < 1 ? 1 : ntiles;
  if (tile >= ntiles) return;
  const int64_t base = tile * kTile + (int64_t)threadIdx.x * ITEMS;
  int32_t v[ITEMS];
  int32_t s = 0;
#pragma unroll
  for (int i = 0; i < ITEMS; ++i) {
    v[i] = (base + i < n) ? load(base + i) : 0;
    s += v[i];
  }
  int32_t agg;
  const int32_t excl = block_scan_excl(s, &agg, wsum);
  if (threadIdx.x < 64) {
    const int32_t prefix = look_back(ss, tile, agg);
    if (threadIdx.x == 0) {
      s_prefix = prefix;
      if (tile == ntiles - 1) finish(prefix + agg);
    }
  }
  __syncthreads();
  int32_t run = s_prefix + excl;
#pragma unroll
  for (int i = 0; i < ITEMS; ++i) {
    if (base + i < n) store(base + i, run, v[i]);
    run += v[i];
  }
}

inline int64_t scan_tiles(int64_t cap, int items) {
  return std::max<int64_t>(1, ceil_div(cap, (int64_t)kThreads * items));
}

// ---------------------------------------------------------------------------
// 0. begin: clear the per-call scan state.  The persistent header holds a
//    magic word, the last finished epoch and the node count the per-node
//    words were built for; if it does not match (first use, another graph
//    size, epochs too close to wrapping around for kChainCalls more calls) the
//    per-node words are cleared and the epochs restart.  Hop h of this call
//    uses epoch top - L + h, where top (header word 2) is written here and
//    becomes the finished epoch at the end of the call.  A chained call skips
//    this launch: the previous call's last step did the same preparation.
// ---------------------------------------------------------------------------
// Fill ranges of the caller done by the same launch (the training step's
// gradient buffers).
struct FillSet {
  int32_t* p[kMaxExtraFills];
  int64_t n[kMaxExtraFills];
  int32_t v[kMaxExtraFills];
  int32_t count;
};

__global__ void __launch_bounds__(kThreads)
begin_kernel(Header* hdr, uint64_t* occ, int64_t N, int32_t L, int32_t* zero, int64_t n_zero,
             FillSet extra) {
  const uint32_t magic = hdr->magic, done = hdr->done_epoch;
  const int64_t n_old = hdr->num_nodes;
  const bool fresh = magic != kMagic || n_old != N || done > 0xFFFFFFFFu - (kChainCalls + 1) * (uint32_t)L;
  const int64_t tid = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  const int64_t stride = (int64_t)gridDim.x * kThreads;
  for (int64_t i = tid; i < n_zero; i += stride) zero[i] = 0;
  for (int r = 0; r < extra.count; ++r)
    for (int64_t i = tid; i < extra.n[r]; i += stride) extra.p[r][i] = extra.v[r];
  if (fresh)
    for (int64_t i = tid; i < N; i += stride) occ[i] = 0;
  if (blockIdx.x == 0 && threadIdx.x == 0) hdr->top_epoch = (fresh ? 0u : done) + (uint32_t)L;
}

// The last launch of a call when no later launch takes it over.
__global__ void __launch_bounds__(kSampleThreads) indices_kernel(SampleTail t) {
  finish_sampling(t, blockIdx.x, gridDim.x, kSampleThreads);
}

// ---------------------------------------------------------------------------
// 1. sample (+ the previous hop's indices in blocks past the sampling grid)
// ---------------------------------------------------------------------------
template <int G, typename RP>
__global__ void __launch_bounds__(kSampleThreads)
sample_kernel(const RP* __restrict__ rowptr, const int32_t* __restrict__ col, int64_t num_nodes,
              const int32_t* __restrict__ dst, const int32_t* n_dst_dev, int32_t cap_dst,
              int32_t* counts, int32_t fanout, uint64_t rng_key, uint32_t hop,
              const Header* hdr, int32_t L, int32_t* __restrict__ nbr_pad,
              int32_t* __restrict__ kcount, uint64_t* __restrict__ occ, int32_t sample_blocks,
              IndexJob prev, TransposeJob tfill, int* err) {
  if ((int32_t)blockIdx.x >= sample_blocks) {
    const int64_t b = blockIdx.x - sample_blocks;
    const int64_t stride = (int64_t)(gridDim.x - sample_blocks) * kSampleThreads;
    index_slots(prev, b * kSampleThreads + threadIdx.x, stride);
    transpose_fill(tfill, b * kSampleThreads + threadIdx.x, stride);
    return;
  }
  const int lane = lane_id();
  const int r = lane & (G - 1);
  // hop 1: the batch (its count is the capacity); later hops: the previous
  // hop's src count, from the device
  int32_t n_dst = n_dst_dev ? *n_dst_dev : cap_dst;
  n_dst = n_dst > cap_dst ? cap_dst : n_dst;
  if (blockIdx.x == 0 && threadIdx.x == 0) counts[0] = n_dst;
  const uint32_t ep = hdr->top_epoch - (uint32_t)L + hop;
  // groups of G lanes, one dst node each; the loop bound is wave-uniform
  constexpr int kPerWave = WAVE / G;
  const int64_t wave = ((int64_t)blockIdx.x * kSampleThreads + threadIdx.x) >> 6;
  const int64_t waves = (int64_t)sample_blocks * (kSampleThreads / 64);
  for (int64_t base = wave * kPerWave; base < n_dst; base += waves * kPerWave) {
    const int64_t i = base + lane / G;
    const bool live = i < n_dst;
    const int32_t v = live ? dst[i] : -1;
    const bool valid = live && v >= 0 && (int64_t)v < num_nodes;
    if (live && !valid && r == 0) set_device_error(err, GNN_DEVERR_SEED_RANGE);
    int32_t w = -1;
    const int32_t k = group_sample<G>(rowptr, col, valid, v, fanout, rng_key, hop, &w);
    if (!live) continue;
    if (r < k && (w < 0 || (int64_t)w >= num_nodes)) {
      set_device_error(err, GNN_DEVERR_GRAPH);
      w = -1;
    }
    if (r == 0) {
      kcount[i] = k;
      if (valid) atomicMax(reinterpret_cast<unsigned long long*>(&occ[v]), occ_word(ep, i));
    }
    if (r < fanout) nbr_pad[i * (int64_t)fanout + r] = w;
    if (r < k && w >= 0)
      atomicMax(reinterpret_cast<unsigned long long*>(&occ[w]),
                occ_word(ep, n_dst + i * (int64_t)fanout + r));
  }
}

// ---------------------------------------------------------------------------
// 2. scans: blocks [0, count_blocks) scan the per-node counts into indptr
//    (counts[2] = E); the others scan the first-occurrence flags into local
//    ids (counts[1] = n_src) and emit src_nodes, src_occ and the per-node id.
// ---------------------------------------------------------------------------
__device__ __forceinline__ int32_t key_at(int64_t pos, int32_t n_dst, const int32_t* dst,
                                          const int32_t* nbr_pad) {
  return pos < n_dst ? dst[pos] : nbr_pad[pos - n_dst];
}

//    Blocks past count_blocks + flag_blocks scan the previous hop's per-src
//    edge counts into its transpose's list offsets (if tr.t_ptr is set).
template <int ITEMS>
__global__ void __launch_bounds__(kThreads)
scans_kernel(const int32_t* __restrict__ dst, const int32_t* __restrict__ nbr_pad, int32_t* counts,
             int32_t fanout, const int32_t* __restrict__ kcount, int32_t* __restrict__ indptr,
             int32_t count_blocks, int32_t flag_blocks, const uint64_t* __restrict__ occ,
             const Header* hdr, int32_t L, uint32_t hop, int64_t num_nodes,
             int32_t* __restrict__ nid, int32_t cap_src, int32_t* __restrict__ src_nodes,
             int32_t* __restrict__ src_occ, ScanState s_cnt, ScanState s_flag, ScanState s_tr,
             TransposeJob tr, int32_t use_ticket, int* err) {
  // (signed throughout: -1 asks tile_scan for a ticket)
  const int32_t bid = (int32_t)blockIdx.x;
  if (bid >= count_blocks + flag_blocks) {
    const int64_t tile = use_ticket ? int64_t{-1} : (int64_t)(bid - count_blocks - flag_blocks);
    const int32_t nd = tr.counts[0];
    auto load = [&](int64_t u) -> int32_t {
      const int32_t c = tr.src_occ[u] - (u < nd ? 1 : 0);
      return c > 0 ? c : 0;
    };
    auto store = [&](int64_t u, int32_t pre, int32_t) {
      tr.t_ptr[u] = pre;
      tr.t_cur[u] = pre;
    };
    const int32_t ns = tr.counts[1];
    auto finish = [&](int32_t total) { tr.t_ptr[ns] = total; };
    tile_scan<ITEMS>(s_tr, tile, ns, load, store, finish);
    return;
  }
  const int32_t n_dst = counts[0];
  const int64_t tile = use_ticket ? int64_t{-1} : (int64_t)(bid < count_blocks ? bid : bid - count_blocks);
  if ((int32_t)blockIdx.x < count_blocks) {
    auto load = [&](int64_t i) -> int32_t { return kcount[i]; };
    auto store = [&](int64_t i, int32_t pre, int32_t) { indptr[i] = pre; };
    auto finish = [&](int32_t total) {
      indptr[n_dst] = total;
      counts[2] = total;
    };
    tile_scan<ITEMS>(s_cnt, tile, n_dst, load, store, finish);
    return;
  }
  const uint32_t ep = hdr->top_epoch - (uint32_t)L + hop;
  const int64_t n = (int64_t)n_dst * (1 + fanout);
  // the dst nodes (distinct) always keep their positions as ids
  auto load = [&](int64_t i) -> int32_t {
    if (i < n_dst) return 1;
    const int32_t key = nbr_pad[i - n_dst];
    if (key < 0) return 0;
    return occ[key] == occ_word(ep, i) ? 1 : 0;
  };
  auto store = [&](int64_t i, int32_t id, int32_t f) {
    if (!f) return;
    if (id < cap_src) {
      const int32_t key = key_at(i, n_dst, dst, nbr_pad);
      src_nodes[id] = key;
      src_occ[id] = i < n_dst ? 1 : 0;
      if (key >= 0 && (int64_t)key < num_nodes) nid[key] = id;
    } else {
      set_device_error(err, GNN_DEVERR_CAPACITY);
    }
  };
  auto finish = [&](int32_t total) { counts[1] = total; };
  tile_scan<ITEMS>(s_flag, tile, n, load, store, finish);
}

}  // namespace

// Scratch layout of one gnn_sample_blocks call.  Persistent part (kept
// between calls, laid out from N alone): the header, the per-node
// first-occurrence words and two per-node local-id tables (hops alternate).  Per call: tickets and scan
// status (cleared by the begin launch), per-hop counts, two padded edge
// buffers (hops alternate).
struct SampleScratch {
  Header* hdr;
  uint64_t* occ;                         // [N]
  int32_t* nid[2];                       // [N] each
  int32_t* tickets;                      // [3 L]
  uint64_t* status[3 * GNN_MAX_LAYERS];  // scan tile status (counts, flags, transposed counts)
  void* zero_begin;                      // [zero_begin, zero_end): cleared once per call
  void* zero_end;
  int32_t* kcount[GNN_MAX_LAYERS];       // [cap_dst]
  int32_t* nbr_pad[2];                   // [max cap_edges]
};

static size_t carve_sample(Carver& c, const int32_t* cap_dst, const int32_t* cap_src,
                           const int64_t* cap_edges, int32_t L, int64_t N, SampleScratch* s) {
  s->hdr = c.take<Header>(1);
  s->occ = c.take<uint64_t>(std::max<int64_t>(1, N));
  s->nid[0] = c.take<int32_t>(std::max<int64_t>(1, N));
  s->nid[1] = c.take<int32_t>(std::max<int64_t>(1, N));
  s->zero_begin = c.take<char>(0);
  s->tickets = c.take<int32_t>(3 * GNN_MAX_LAYERS);
  for (int h = 0; h < L; ++h) {
    s->status[3 * h] = c.take<uint64_t>(scan_tiles(cap_dst[h], kScanItemsMin));
    s->status[3 * h + 1] =
        c.take<uint64_t>(scan_tiles((int64_t)cap_dst[h] + cap_edges[h], kScanItemsMin));
    s->status[3 * h + 2] = c.take<uint64_t>(scan_tiles(cap_src[h], kScanItemsMin));
  }
  s->zero_end = c.take<char>(0);
  int64_t max_edges = 1;
  for (int h = 0; h < L; ++h) {
    s->kcount[h] = c.take<int32_t>(std::max<int64_t>(1, cap_dst[h]));
    max_edges = std::max<int64_t>(max_edges, cap_edges[h]);
  }
  s->nbr_pad[0] = c.take<int32_t>(max_edges);
  s->nbr_pad[1] = c.take<int32_t>(max_edges);
  return c.off;
}

size_t sample_scratch_bytes(const int32_t* cap_dst, const int32_t* cap_src,
                            const int64_t* cap_edges, int32_t L, int64_t N) {
  Carver c(nullptr, 0);
  SampleScratch s;
  return carve_sample(c, cap_dst, cap_src, cap_edges, L, N, &s);
}

template <typename RP>
static int sample_hops(const gnn_csr* csr, const RP* rowptr, const int32_t* seeds, int32_t B,
                       const int32_t* fanouts, int32_t L, uint64_t rng_key, gnn_block* blocks,
                       void* ws, size_t ws_bytes, const FillRange* extra, int n_extra,
                       SampleTail* tail, const BlockTranspose* tr, hipStream_t st, bool chained) {
  if (n_extra < 0 || n_extra > kMaxExtraFills) return fail(GNN_EINVAL, "sampler: too many fills");
  if (int rc = check_csr_options(csr, "sampler")) return rc;
  int32_t cap_dst[GNN_MAX_LAYERS], cap_src[GNN_MAX_LAYERS];
  int64_t cap_edges[GNN_MAX_LAYERS];
  for (int h = 0; h < L; ++h) {
    cap_src[h] = blocks[h].cap_src;
    cap_dst[h] = blocks[h].cap_dst;
    cap_edges[h] = blocks[h].cap_edges;
    if (cap_edges[h] != (int64_t)cap_dst[h] * fanouts[h])
      return fail(GNN_EINVAL, "gnn_sample_blocks: cap_edges must equal cap_dst * fanout");
  }
  const int64_t N = csr->num_nodes;
  Carver c(ws, ws_bytes);
  SampleScratch sc;
  carve_sample(c, cap_dst, cap_src, cap_edges, L, N, &sc);
  if (!c.fits()) return fail(GNN_EWORKSPACE, "gnn_sample_blocks: workspace %zu < %zu bytes", ws_bytes, c.off);
  int* err = device_error_word();
  if (!err) return fail(GNN_EHIP, "device error word unavailable");

  const int64_t zero_words =
      (static_cast<char*>(sc.zero_end) - static_cast<char*>(sc.zero_begin)) / 4;
  FillSet fs{};
  for (int r = 0; r < n_extra; ++r) {
    fs.p[r] = static_cast<int32_t*>(extra[r].p);
    fs.n[r] = extra[r].p ? extra[r].n_words : 0;
    fs.v[r] = extra[r].value;
  }
  fs.count = n_extra;
  if (blocks[0].cap_dst != B) return fail(GNN_EINVAL, "sampler: hop 1 capacity %d != batch %d", blocks[0].cap_dst, B);
  if (!chained || n_extra > 0)
    launch("begin", begin_kernel, kBeginBlocks, kThreads, 0, st, sc.hdr, sc.occ, N, L,
           static_cast<int32_t*>(sc.zero_begin), zero_words, fs);

  // transposes (hops h < L - 1, if asked for): hop h's counts are scanned in
  // hop h + 1's scans launch and its lists filled by the launch after it
  auto tjob = [&](int h) -> TransposeJob {
    TransposeJob t{};
    if (!tr || h < 0 || h >= L - 1 || !tr[h].t_ptr) return t;
    const gnn_block& b = blocks[h];
    t = TransposeJob{b.indptr, b.indices, b.counts, b.src_occ, tr[h].t_ptr, tr[h].t_cur,
                     tr[h].t_dst, fanouts[h], b.cap_src};
    return t;
  };
  IndexJob prev{};
  int64_t prev_slots = 0;
  for (int h = 0; h < L; ++h) {
    gnn_block& bk = blocks[h];
    const int32_t* dst = h == 0 ? seeds : blocks[h - 1].src_nodes;
    const int32_t* n_dst_src = h == 0 ? nullptr : blocks[h - 1].counts + 1;
    const int32_t f = fanouts[h];
    int32_t* pad = sc.nbr_pad[h & 1];
    int32_t* nid = sc.nid[h & 1];

    // lanes per dst node: the whole wave (scalar broadcasts) while one wave
    // per node fits the resident waves of the GPU, else the smallest group
    // that holds the fanout (4 or 2 nodes per wave)
    int G = 64;
    if ((int64_t)bk.cap_dst > kResidentWaves) G = f <= 16 ? 16 : (f <= 32 ? 32 : 64);
    const int64_t per_block = (kSampleThreads / 64) * (64 / G);
    const int64_t sblocks = std::min<int64_t>(kSampleMaxBlocks,
                                              std::max<int64_t>(1, ceil_div(bk.cap_dst, per_block)));
    // extra blocks: hop h - 1's compaction and hop h - 2's transpose fill
    const TransposeJob tfill = tjob(h - 2);
    const int64_t extra_slots = std::max<int64_t>(prev_slots, tfill.t_dst ? blocks[h - 2].cap_edges : 0);
    const int64_t iblocks =
        h == 0 ? 0
               : std::min<int64_t>(kIndexBlocksMax,
                                   std::max<int64_t>(1, ceil_div(extra_slots, kSampleThreads * 4)));
    const unsigned grid = (unsigned)(sblocks + iblocks);
    auto go = [&](auto kernel) {
      launch("sample", kernel, grid, kSampleThreads, 0, st, rowptr, csr->col, N, dst, n_dst_src,
             bk.cap_dst, bk.counts, f, rng_key, (uint32_t)(h + 1), sc.hdr, L, pad, sc.kcount[h],
             sc.occ, (int32_t)sblocks, prev, tfill, err);
    };
    if (G == 16) go(sample_kernel<16, RP>);
    else if (G == 32) go(sample_kernel<32, RP>);
    else go(sample_kernel<64, RP>);
    ScanState s_cnt{sc.tickets + 3 * h, sc.status[3 * h], err};
    ScanState s_flag{sc.tickets + 3 * h + 1, sc.status[3 * h + 1], err};
    // hop h - 1's transposed counts (its compaction ran in this hop's sample launch)
    const TransposeJob tscan = tjob(h - 1);
    ScanState s_tr{sc.tickets + 3 * h + 2, h >= 1 ? sc.status[3 * (h - 1) + 2] : nullptr, err};
    // a grid that is resident all at once can number its tiles by block id;
    // a larger one takes tickets, so that a tile only waits on running tiles
    int items = kScanItemsMin;
    auto tr_tiles = [&](int it) -> int64_t {
      return tscan.t_ptr ? scan_tiles(blocks[h - 1].cap_src, it) : 0;
    };
    auto tiles = [&](int it) {
      return scan_tiles(bk.cap_dst, it) + scan_tiles((int64_t)bk.cap_dst + bk.cap_edges, it) +
             tr_tiles(it);
    };
    while (items < kScanItemsMax && tiles(items) > kResidentScanBlocks) items *= 2;
    const int64_t cb = scan_tiles(bk.cap_dst, items);
    const int64_t fb = scan_tiles((int64_t)bk.cap_dst + bk.cap_edges, items);
    // tiles numbered by block id when the grid is resident at once, tickets
    // otherwise or when the graph's options ask for them (same blocks)
    const int32_t use_ticket = (csr->scan_order == 1 || tiles(items) > kResidentScanBlocks) ? 1 : 0;
    auto scan = [&](auto kernel) {
      launch("scans", kernel, (unsigned)tiles(items), kThreads, 0, st, dst, pad, bk.counts, f,
             sc.kcount[h], bk.indptr, (int32_t)cb, (int32_t)fb, sc.occ, sc.hdr, L,
             (uint32_t)(h + 1), N, nid, bk.cap_src, bk.src_nodes, bk.src_occ, s_cnt, s_flag, s_tr,
             tscan, use_ticket, err);
    };
    if (items == 2) scan(scans_kernel<2>);
    else if (items == 4) scan(scans_kernel<4>);
    else scan(scans_kernel<8>);
    GNN_LAUNCH_CHECK("gnn_sample_blocks");
    prev = IndexJob{pad, sc.kcount[h], bk.indptr, bk.counts, nid, bk.indices, bk.src_occ, f, bk.cap_src, N};
    prev_slots = bk.cap_edges;
  }
  // the last step: the last hop's compaction and hop L - 2's transpose fill
  const SampleTail last{prev, sc.hdr, tjob(L - 2), static_cast<int32_t*>(sc.zero_begin), zero_words,
                        (uint32_t)L};
  if (tail) {  // the caller's next launch finishes the call
    *tail = last;
    return GNN_OK;
  }
  const int64_t tail_slots = std::max<int64_t>(prev_slots, last.tfill.t_dst ? blocks[L - 2].cap_edges : 0);
  const int64_t gx = std::min<int64_t>(kIndexBlocksMax, std::max<int64_t>(1, ceil_div(tail_slots, kSampleThreads * 4)));
  launch("indices", indices_kernel, (unsigned)gx, kSampleThreads, 0, st, last);
  GNN_LAUNCH_CHECK("gnn_sample_blocks indices");
  return GNN_OK;
}

int sample_blocks_impl(const gnn_csr* csr, const int32_t* seeds, int32_t B, const int32_t* fanouts,
                       int32_t L, uint64_t rng_key, gnn_block* blocks, void* ws, size_t ws_bytes,
                       const FillRange* extra, int n_extra, SampleTail* tail, hipStream_t st,
                       const BlockTranspose* tr, bool chained) {
  if (csr->rowptr_bits == 64)
    return sample_hops(csr, static_cast<const int64_t*>(csr->rowptr), seeds, B, fanouts, L, rng_key,
                       blocks, ws, ws_bytes, extra, n_extra, tail, tr, st, chained);
  return sample_hops(csr, static_cast<const int32_t*>(csr->rowptr), seeds, B, fanouts, L, rng_key,
                     blocks, ws, ws_bytes, extra, n_extra, tail, tr, st, chained);
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
  return gnn::sample_scratch_bytes(cd, cs, ce, L, N);
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
  if (int rc = check_csr_options(csr, "gnn_sample_blocks")) return rc;
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
  if (ws_bytes < sample_scratch_bytes(cd, cs, ce, L, csr->num_nodes))
    return fail(GNN_EWORKSPACE, "gnn_sample_blocks: workspace too small");
  // the kernels size their grids from the capacities given in `blocks`
  gnn_block local[GNN_MAX_LAYERS];
  for (int h = 0; h < L; ++h) {
    local[h] = blocks[h];
    local[h].cap_dst = cd[h];
    local[h].cap_src = blocks[h].cap_src;
    local[h].cap_edges = ce[h];
  }
  return sample_blocks_impl(csr, seeds, B, fanouts, L, rng_key, local, ws, ws_bytes, nullptr, 0,
                            nullptr, as_stream(stream));
}

}  // extern "C"
