// Layer-wise neighbour sampling and block construction.
//
// Per hop h (Neighbor Sampling, paper section 2.2; budgets of section 5.1.2):
//   1. count:   k_i = min(fanout, deg(dst_i))                (one thread per dst)
//   2. scan:    indptr = exclusive prefix sum of k
//   3. sample:  one wavefront per dst node; Floyd's algorithm over CSR
//               positions driven by Philox4x64-10 keyed by (rng_key, hop, node);
//               the picks are ranked across the wave and the neighbours written
//               in ascending position order.
//   4. relabel: dst list ++ sampled ids -> local ids in first-occurrence order.
//               Keys are hash-partitioned so that every partition fits an LDS
//               open-addressing table; each table records, per key, the minimum
//               position (atomicMin) and the number of occurrences.  Flags
//               "position == first position" are scanned into local ids.  The
//               result does not depend on thread scheduling.
#include "internal.hpp"
#include "philox.hpp"
#include "wave.hpp"

namespace gnn {

namespace {

constexpr int kThreads = 256;
constexpr int kTableSlots = 4096;        // LDS table entries per partition
constexpr int kTableBits = 12;
constexpr int kTargetPerPart = 2048;     // average elements per partition (upper bound)
constexpr int kMaxParts = 4096;
constexpr int32_t kEmpty = -1;

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

template <typename RP>
__device__ __forceinline__ void row_range(const RP* rowptr, int32_t v, int64_t& start, int64_t& deg) {
  start = (int64_t)rowptr[v];
  deg = (int64_t)rowptr[v + 1] - start;
}

// ---------------------------------------------------------------------------
// 1. count
// ---------------------------------------------------------------------------
template <typename RP>
__global__ void __launch_bounds__(kThreads)
count_kernel(const RP* __restrict__ rowptr, int64_t num_nodes, const int32_t* __restrict__ dst,
             const int32_t* n_src_dev, int32_t cap_dst, int32_t fanout, int32_t* n_dst_out,
             int32_t* __restrict__ k_out, int* err) {
  int32_t n = *n_src_dev;
  n = n > cap_dst ? cap_dst : n;
  const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (i == 0) *n_dst_out = n;
  if (i >= n) return;
  const int32_t v = dst[i];
  int32_t k = 0;
  if (v < 0 || (int64_t)v >= num_nodes) {
    set_device_error(err, GNN_DEVERR_SEED_RANGE);
  } else {
    int64_t s, d;
    row_range(rowptr, v, s, d);
    k = (int32_t)(d < fanout ? d : fanout);
  }
  k_out[i] = k;
}

// ---------------------------------------------------------------------------
// 3. sample: one wavefront per dst node
// ---------------------------------------------------------------------------
template <typename RP>
__global__ void __launch_bounds__(kThreads)
sample_kernel(const RP* __restrict__ rowptr, const int32_t* __restrict__ col, int64_t num_nodes,
              const int32_t* __restrict__ dst, const int32_t* n_dst_dev,
              const int32_t* __restrict__ indptr, int32_t fanout, uint64_t rng_key, uint32_t hop,
              int32_t* __restrict__ nbr) {
  const int lane = lane_id();
  const int64_t i = ((int64_t)blockIdx.x * kThreads + threadIdx.x) >> 6;
  if (i >= *n_dst_dev) return;
  const int32_t v = dst[i];
  if (v < 0 || (int64_t)v >= num_nodes) return;
  int64_t start, d;
  row_range(rowptr, v, start, d);
  int32_t* out = nbr + indptr[i];
  if (d <= fanout) {
    if (lane < d) out[lane] = col[start + lane];
    return;
  }
  const uint32_t du = (uint32_t)d;
  const uint32_t f = (uint32_t)fanout;
  // lane s computes t_s = uniform in [0, j_s], j_s = d - f + s
  uint32_t t = 0;
  if ((uint32_t)lane < f) {
    const uint64_t r = sample_draw(rng_key, hop, (uint32_t)v, (uint32_t)lane);
    t = bounded_draw(r, du - f + (uint32_t)lane + 1u);
  }
  // Floyd: step s keeps t_s unless an earlier step already chose it, then j_s.
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
  if ((uint32_t)lane < f) out[rank] = col[start + pick];
}

// ---------------------------------------------------------------------------
// 4. relabel
// ---------------------------------------------------------------------------
struct RelabelBufs {
  int32_t* hist;        // [kMaxParts]
  int32_t* part_start;  // [kMaxParts + 1]
  int32_t* cursor;      // [kMaxParts]
  int32_t* buf_key;     // [cap_total]
  int32_t* buf_pos;     // [cap_total]
  int32_t* first;       // [cap_total]
  int32_t* flag;        // [cap_total]
  int32_t* occ;         // [cap_total]
  int32_t* newid;       // [cap_total + 1]
  int32_t* gkey;        // [2 * cap_total] fallback tables
  int32_t* gmin;        // [2 * cap_total]
  int32_t* gcnt;        // [2 * cap_total]
  int32_t* total;       // [1] n_dst + E
};

__device__ __forceinline__ int32_t key_at(int64_t pos, int32_t n_dst, const int32_t* dst,
                                          const int32_t* nbr) {
  return pos < n_dst ? dst[pos] : nbr[pos - n_dst];
}

constexpr int kItems = 8;
constexpr int kTile = kThreads * kItems;

// total = n_dst + E for the later kernels
__global__ void total_kernel(const int32_t* counts, int32_t* total) {
  if (threadIdx.x == 0 && blockIdx.x == 0) *total = counts[0] + counts[2];
}

__global__ void __launch_bounds__(kThreads)
hist_kernel(const int32_t* __restrict__ dst, const int32_t* __restrict__ nbr,
            const int32_t* counts, int log_parts, int32_t* __restrict__ hist) {
  __shared__ int32_t lh[kMaxParts];
  const int parts = 1 << log_parts;
  const int32_t n_dst = counts[0];
  const int64_t total = (int64_t)n_dst + counts[2];
  const int64_t base = (int64_t)blockIdx.x * kTile;
  if (base >= total) return;
  for (int p = threadIdx.x; p < parts; p += kThreads) lh[p] = 0;
  __syncthreads();
#pragma unroll
  for (int it = 0; it < kItems; ++it) {
    const int64_t pos = base + (int64_t)it * kThreads + threadIdx.x;
    if (pos < total) atomicAdd(&lh[part_of(key_at(pos, n_dst, dst, nbr), log_parts)], 1);
  }
  __syncthreads();
  for (int p = threadIdx.x; p < parts; p += kThreads)
    if (lh[p]) atomicAdd(&hist[p], lh[p]);
}

__global__ void __launch_bounds__(1024)
part_scan_kernel(int32_t* hist, int log_parts, int32_t* part_start, int32_t* cursor) {
  __shared__ int32_t wsum[16];
  __shared__ int32_t carry;
  const int parts = 1 << log_parts;
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  if (threadIdx.x == 0) carry = 0;
  __syncthreads();
  for (int c = 0; c < parts; c += 1024) {
    const int p = c + threadIdx.x;
    const int32_t x = p < parts ? hist[p] : 0;
    const int32_t inc = wave_inclusive_scan(x);
    if (lane == 63) wsum[wid] = inc;
    __syncthreads();
    int32_t off = carry, tot = 0;
    for (int w = 0; w < 16; ++w) {
      off += (w < wid) ? wsum[w] : 0;
      tot += wsum[w];
    }
    if (p < parts) {
      part_start[p] = off + inc - x;
      cursor[p] = off + inc - x;
      hist[p] = 0;  // ready for the next hop
    }
    __syncthreads();
    if (threadIdx.x == 0) carry += tot;
    __syncthreads();
  }
  if (threadIdx.x == 0) part_start[parts] = carry;
}

__global__ void __launch_bounds__(kThreads)
partition_kernel(const int32_t* __restrict__ dst, const int32_t* __restrict__ nbr,
                 const int32_t* counts, int log_parts, int32_t* __restrict__ cursor,
                 int32_t* __restrict__ buf_key, int32_t* __restrict__ buf_pos) {
  __shared__ int32_t lcount[kMaxParts];
  __shared__ int32_t lbase[kMaxParts];
  const int parts = 1 << log_parts;
  const int32_t n_dst = counts[0];
  const int64_t total = (int64_t)n_dst + counts[2];
  const int64_t base = (int64_t)blockIdx.x * kTile;
  if (base >= total) return;
  for (int p = threadIdx.x; p < parts; p += kThreads) lcount[p] = 0;
  __syncthreads();
  int32_t keys[kItems];
  int32_t rank[kItems];
#pragma unroll
  for (int it = 0; it < kItems; ++it) {
    const int64_t pos = base + (int64_t)it * kThreads + threadIdx.x;
    keys[it] = pos < total ? key_at(pos, n_dst, dst, nbr) : 0;
    rank[it] = pos < total ? atomicAdd(&lcount[part_of(keys[it], log_parts)], 1) : 0;
  }
  __syncthreads();
  for (int p = threadIdx.x; p < parts; p += kThreads)
    lbase[p] = lcount[p] ? atomicAdd(&cursor[p], lcount[p]) : 0;
  __syncthreads();
#pragma unroll
  for (int it = 0; it < kItems; ++it) {
    const int64_t pos = base + (int64_t)it * kThreads + threadIdx.x;
    if (pos < total) {
      const int32_t slot = lbase[part_of(keys[it], log_parts)] + rank[it];
      buf_key[slot] = keys[it];
      buf_pos[slot] = (int32_t)pos;
    }
  }
}

// Open-addressing insert / lookup on a table of `cap` slots (power of two when
// in LDS; any size for the global fallback).
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

__global__ void __launch_bounds__(kThreads)
emit_kernel(const int32_t* __restrict__ dst, int32_t* nbr_indices, const int32_t* counts,
            const int32_t* __restrict__ first, const int32_t* __restrict__ flag,
            const int32_t* __restrict__ occ, const int32_t* __restrict__ newid, int32_t cap_src,
            int32_t* __restrict__ src_nodes, int32_t* __restrict__ src_occ, int* err) {
  const int32_t n_dst = counts[0];
  const int64_t total = (int64_t)n_dst + counts[2];
  const int64_t pos = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (pos >= total) return;
  const int32_t key = key_at(pos, n_dst, dst, nbr_indices);
  if (flag[pos]) {
    const int32_t id = newid[pos];
    if (id < cap_src) {
      src_nodes[id] = key;
      src_occ[id] = occ[pos];
    } else {
      set_device_error(err, GNN_DEVERR_CAPACITY);
    }
  }
  if (pos >= n_dst) nbr_indices[pos - n_dst] = newid[first[pos]];
}

struct HopCaps {
  int32_t cap_dst, cap_src;
  int64_t cap_edges;
};

}  // namespace

size_t sample_scratch_bytes(const int32_t* cap_dst, const int32_t* cap_src,
                            const int64_t* cap_edges, int32_t L) {
  int64_t max_total = 1, max_dst = 1;
  for (int h = 0; h < L; ++h) {
    max_total = std::max<int64_t>(max_total, (int64_t)cap_dst[h] + cap_edges[h]);
    max_dst = std::max<int64_t>(max_dst, cap_dst[h]);
  }
  Carver c(nullptr, 0);
  c.take<int32_t>(max_dst);                      // k
  c.take<int32_t>(scan_scratch_ints(std::max(max_dst, max_total)));
  c.take<int32_t>(kMaxParts);                    // hist
  c.take<int32_t>(kMaxParts + 1);                // part_start
  c.take<int32_t>(kMaxParts);                    // cursor
  for (int i = 0; i < 5; ++i) c.take<int32_t>(max_total);
  c.take<int32_t>(max_total + 1);                // newid
  for (int i = 0; i < 3; ++i) c.take<int32_t>(2 * max_total);
  c.take<int32_t>(4);                            // total
  return c.off;
}

template <typename RP>
static int sample_hops(const gnn_csr* csr, const RP* rowptr, const int32_t* seeds, int32_t B,
                       const int32_t* fanouts, int32_t L, uint64_t rng_key, gnn_block* blocks,
                       void* ws, size_t ws_bytes, hipStream_t st) {
  int64_t max_total = 1, max_dst = 1;
  for (int h = 0; h < L; ++h) {
    max_total = std::max<int64_t>(max_total, (int64_t)blocks[h].cap_dst + blocks[h].cap_edges);
    max_dst = std::max<int64_t>(max_dst, blocks[h].cap_dst);
  }
  Carver c(ws, ws_bytes);
  int32_t* kbuf = c.take<int32_t>(max_dst);
  int32_t* scan_scratch = c.take<int32_t>(scan_scratch_ints(std::max(max_dst, max_total)));
  RelabelBufs rb;
  rb.hist = c.take<int32_t>(kMaxParts);
  rb.part_start = c.take<int32_t>(kMaxParts + 1);
  rb.cursor = c.take<int32_t>(kMaxParts);
  rb.buf_key = c.take<int32_t>(max_total);
  rb.buf_pos = c.take<int32_t>(max_total);
  rb.first = c.take<int32_t>(max_total);
  rb.flag = c.take<int32_t>(max_total);
  rb.occ = c.take<int32_t>(max_total);
  rb.newid = c.take<int32_t>(max_total + 1);
  rb.gkey = c.take<int32_t>(2 * max_total);
  rb.gmin = c.take<int32_t>(2 * max_total);
  rb.gcnt = c.take<int32_t>(2 * max_total);
  rb.total = c.take<int32_t>(4);
  if (!c.fits()) return fail(GNN_EWORKSPACE, "gnn_sample_blocks: workspace %zu < %zu bytes", ws_bytes, c.off);
  int* err = device_error_word();
  if (!err) return fail(GNN_EHIP, "device error word unavailable");

  // hop 1's dst count lives in blocks[0].counts[0]; zero the partition histogram
  FillRange fr[2] = {{blocks[0].counts, 1, B}, {rb.hist, kMaxParts, 0}};
  if (int rc = launch_fill(fr, 2, st)) return rc;

  for (int h = 0; h < L; ++h) {
    gnn_block& bk = blocks[h];
    const int32_t* dst = h == 0 ? seeds : blocks[h - 1].src_nodes;
    const int32_t* n_dst_src = h == 0 ? blocks[0].counts : blocks[h - 1].counts + 1;
    const int32_t f = fanouts[h];
    const int64_t cap_total = (int64_t)bk.cap_dst + bk.cap_edges;
    const int parts = partitions_for(cap_total);
    const int lp = log2i(parts);

    unsigned gb = (unsigned)std::max<int64_t>(1, ceil_div(bk.cap_dst, kThreads));
    count_kernel<RP><<<gb, kThreads, 0, st>>>(rowptr, csr->num_nodes, dst, n_dst_src, bk.cap_dst, f,
                                              bk.counts, kbuf, err);
    if (int rc = launch_exclusive_scan(kbuf, bk.indptr, bk.counts, bk.cap_dst, bk.counts + 2,
                                       scan_scratch, st))
      return rc;
    unsigned gs = (unsigned)std::max<int64_t>(1, ceil_div((int64_t)bk.cap_dst * 64, kThreads));
    sample_kernel<RP><<<gs, kThreads, 0, st>>>(rowptr, csr->col, csr->num_nodes, dst, bk.counts,
                                               bk.indptr, f, rng_key, (uint32_t)(h + 1), bk.indices);
    unsigned gt = (unsigned)std::max<int64_t>(1, ceil_div(cap_total, kTile));
    hist_kernel<<<gt, kThreads, 0, st>>>(dst, bk.indices, bk.counts, lp, rb.hist);
    part_scan_kernel<<<1, 1024, 0, st>>>(rb.hist, lp, rb.part_start, rb.cursor);
    partition_kernel<<<gt, kThreads, 0, st>>>(dst, bk.indices, bk.counts, lp, rb.cursor, rb.buf_key,
                                              rb.buf_pos);
    table_kernel<<<parts, kThreads, 0, st>>>(rb.part_start, rb.buf_key, rb.buf_pos, rb.first,
                                             rb.flag, rb.occ, rb.gkey, rb.gmin, rb.gcnt);
    total_kernel<<<1, 64, 0, st>>>(bk.counts, rb.total);
    if (int rc = launch_exclusive_scan(rb.flag, rb.newid, rb.total, cap_total, bk.counts + 1,
                                       scan_scratch, st))
      return rc;
    unsigned ge = (unsigned)std::max<int64_t>(1, ceil_div(cap_total, kThreads));
    emit_kernel<<<ge, kThreads, 0, st>>>(dst, bk.indices, bk.counts, rb.first, rb.flag, rb.occ,
                                         rb.newid, bk.cap_src, bk.src_nodes, bk.src_occ, err);
    GNN_LAUNCH_CHECK("gnn_sample_blocks");
  }
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
