// ShaDow k-hop localised subgraphs (paper section 2.2, ShaDow K-Hop Sampling;
// section 5.2): per root, a breadth-first neighbour-sampled node set, then all
// edges of the graph among that set (the induced subgraph).  The batch is the
// disjoint union of the roots' subgraphs as one square block, numbered roots
// first: root r has local id r, then each component's other nodes follow,
// component after component, in first-occurrence order; rows list their
// induced neighbours in ascending global id.
//
// Three kernels:
//   build: one workgroup per root.  Hop by hop, each wave samples frontier
//          nodes (same sampler and Philox stream as layer-wise sampling); new
//          nodes are appended in first-occurrence order using two LDS hash
//          tables (the node set, and the first candidate position of each key
//          of the hop).  Then each wave scans the CSR rows of the set's nodes
//          and keeps the neighbours found in the LDS node table.  Per-root
//          nodes, row counts and edges go to a staging area.
//   scan:  one workgroup: prefix sums of the per-root counts.
//   emit:  one workgroup per root writes its rows into the final block.
#include <atomic>

#include "internal.hpp"
#include "sampler.hpp"
#include "wave.hpp"

namespace gnn {

namespace {

constexpr int kThreads = 512;
constexpr int kWaves = kThreads / 64;
constexpr int32_t kEmpty = -1;
constexpr int kBitmapCap = 512;   // node sets up to this size use the LDS bitmap
// Degree above which a subgraph node's CSR row is searched, not read whole
// (node sets up to kBitmapCap), unless the graph's options give another; the
// output does not depend on it
constexpr int32_t kHubDegree = 1024;
constexpr int kChunkBatch = 16;   // 64-element row chunks in flight per lane
constexpr int kFilterLog2 = 15;   // node-set filter: 2^15 bits (4 KB of LDS)
constexpr int kFilterBits = 1 << kFilterLog2;

inline int64_t shadow_max_nodes(int32_t fanout, int32_t hops) {
  int64_t n = 1, p = 1;
  for (int h = 0; h < hops; ++h) {
    p *= fanout;
    n += p;
  }
  return n;
}

__device__ __forceinline__ uint32_t hslot(int32_t key) {
  uint32_t h = (uint32_t)key * 0x9E3779B1u;
  return h ^ (h >> 16);
}

// Bit of a key in the node-set filter (independent of hslot).
__device__ __forceinline__ uint32_t fslot(int32_t key) {
  return ((uint32_t)key * 0x85EBCA6Bu) >> (32 - kFilterLog2);
}

// LDS hash (key -> value), `cap` a power of two, linear probing.
__device__ __forceinline__ void h_insert_min(int32_t* hk, int32_t* hv, uint32_t cap, int32_t key,
                                             int32_t val) {
  uint32_t s = hslot(key) & (cap - 1);
  while (true) {
    const int32_t old = atomicCAS(&hk[s], kEmpty, key);
    if (old == kEmpty || old == key) {
      atomicMin(&hv[s], val);
      return;
    }
    s = (s + 1) & (cap - 1);
  }
}

__device__ __forceinline__ int32_t h_find(const int32_t* hk, const int32_t* hv, uint32_t cap,
                                          int32_t key) {
  uint32_t s = hslot(key) & (cap - 1);
  while (true) {
    const int32_t k = hk[s];
    if (k == key) return hv[s];
    if (k == kEmpty) return -1;
    s = (s + 1) & (cap - 1);
  }
}

__device__ __forceinline__ int32_t block_excl_scan(int32_t x, int32_t* total, int32_t* wsum) {
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const int32_t inc = wave_inclusive_scan(x);
  if (lane == 63) wsum[wid] = inc;
  __syncthreads();
  int32_t off = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    off += (w < wid) ? wsum[w] : 0;
    tot += wsum[w];
  }
  __syncthreads();
  *total = tot;
  return off + inc - x;
}

struct ShadowStage {
  int32_t* nodes;    // [B x NMAX] global ids, component order
  int32_t* rowcnt;   // [B x NMAX] induced degree per component node
  int32_t* edges;    // [B x NMAX x (NMAX - 1)] component-local neighbour index
  int32_t* per_root; // [B x 4]: nodes, root-row edges, other-row edges, 0
};

// NCAP: LDS capacity in nodes (>= max nodes per root and >= candidates per hop).
template <int NCAP, typename RP>
__global__ void __launch_bounds__(kThreads)
shadow_build_kernel(const RP* __restrict__ rowptr, const int32_t* __restrict__ col,
                    int64_t num_nodes, const int32_t* __restrict__ roots, int32_t B, int32_t fanout,
                    int32_t hops, uint64_t rng_key, int32_t nmax, ShadowStage stg, int* err,
                    int32_t hub_deg) {
  constexpr int HCAP = 2 * NCAP;  // power of two (NCAP is)
  __shared__ int32_t nodes[NCAP];
  __shared__ int32_t nk[HCAP], nv[HCAP];  // node set: global id -> component index
  __shared__ int32_t cand[NCAP];
  __shared__ int32_t ck[HCAP], cv[HCAP];  // this hop: key -> first candidate position
  __shared__ int32_t wsum[kWaves];
  __shared__ int32_t s_n, s_fb, s_fe;
  const int r = blockIdx.x;
  if (r >= B) return;
  const int lane = lane_id(), wave = threadIdx.x >> 6;
  for (int i = threadIdx.x; i < HCAP; i += kThreads) {
    nk[i] = kEmpty;
    nv[i] = 0x7FFFFFFF;
  }
  __syncthreads();
  const int32_t root = roots[r];
  const bool root_ok = root >= 0 && (int64_t)root < num_nodes;
  if (threadIdx.x == 0) {
    if (!root_ok) set_device_error(err, GNN_DEVERR_SEED_RANGE);
    nodes[0] = root;
    h_insert_min(nk, nv, HCAP, root, 0);
    s_n = 1;
    s_fb = 0;
    s_fe = 1;
  }
  __syncthreads();
  for (int32_t h = 1; h <= hops && root_ok; ++h) {
    const int32_t fb = s_fb, fe = s_fe;
    const int32_t ncand = (fe - fb) * fanout;  // <= NCAP by construction
    for (int i = threadIdx.x; i < HCAP; i += kThreads) {
      ck[i] = kEmpty;
      cv[i] = 0x7FFFFFFF;
    }
    // sample every frontier node (one wave per node); candidates keep
    // (frontier order, ascending position) order
    for (int32_t j = fb + wave; j < fe; j += kWaves) {
      int32_t w = -1;
      wave_sample(rowptr, col, nodes[j], fanout, rng_key, (uint32_t)h, &w);
      if (lane < fanout) cand[(j - fb) * fanout + lane] = w;
    }
    __syncthreads();
    for (int32_t c = threadIdx.x; c < ncand; c += kThreads)
      if (cand[c] >= 0) h_insert_min(ck, cv, HCAP, cand[c], c);
    __syncthreads();
    // a candidate joins the set if it is the first occurrence of its key in
    // this hop and not already in the set
    const int32_t n0 = s_n;
    int32_t base = n0;
    for (int32_t c0 = 0; c0 < ncand; c0 += kThreads) {
      const int32_t c = c0 + threadIdx.x;
      int32_t is_new = 0, key = -1;
      if (c < ncand) {
        key = cand[c];
        is_new = key >= 0 && h_find(ck, cv, HCAP, key) == c && h_find(nk, nv, HCAP, key) < 0;
      }
      int32_t tot;
      const int32_t off = block_excl_scan(is_new, &tot, wsum);
      if (is_new) {
        nodes[base + off] = key;
        h_insert_min(nk, nv, HCAP, key, base + off);
      }
      base += tot;
      __syncthreads();
    }
    if (threadIdx.x == 0) {
      s_fb = n0;
      s_fe = base;
      s_n = base;
    }
    __syncthreads();
  }
  const int32_t n = s_n;
  int32_t* gnodes = stg.nodes + (int64_t)r * nmax;
  int32_t* grow = stg.rowcnt + (int64_t)r * nmax;
  int32_t* gedge = stg.edges + (int64_t)r * nmax * (nmax - 1);
  for (int i = threadIdx.x; i < n; i += kThreads) gnodes[i] = nodes[i];
  int32_t e_root = 0, e_other = 0;
  if constexpr (NCAP <= kBitmapCap) {
    // induced edges: the CSR rows of all set nodes are read in 64-element
    // chunks spread over the waves, kChunkBatch chunks in flight per lane; a
    // neighbour found in the node set sets bit (i, j) of an n x n bitmap.
    // Rows are then written in ascending global id of the neighbour.
    constexpr int W = NCAP / 32;  // bitmap words per row
    __shared__ int64_t rstart[NCAP];
    __shared__ int32_t rdeg[NCAP];
    __shared__ int32_t cpre[NCAP + 1];
    __shared__ int32_t ord[NCAP];
    __shared__ uint32_t bits[NCAP * W];
    // one-hash bit filter of the node set: almost every row element is not in
    // the set, and the filter rejects it with one LDS read instead of a probe
    // sequence of the hash table
    __shared__ uint32_t filt[kFilterBits / 32];
    for (int i = threadIdx.x; i < NCAP * W; i += kThreads) bits[i] = 0;
    for (int i = threadIdx.x; i < kFilterBits / 32; i += kThreads) filt[i] = 0;
    __syncthreads();
    for (int i = threadIdx.x; i < n; i += kThreads) {
      const uint32_t b = fslot(nodes[i]);
      atomicOr(&filt[b >> 5], 1u << (b & 31));
    }
    // Rows longer than hub_deg ("hubs") are not read whole.  The graph is
    // symmetric, so an induced edge with a non-hub endpoint is found from
    // that endpoint's row and both of its bits are set; an edge between two
    // hubs is found by a binary search of one hub's id in the other's
    // (sorted, shorter) row.
    auto row_chunks = [&](int64_t d) { return d > hub_deg ? 0 : (int32_t)((d + 63) / 64); };
    int32_t chunks = 0;
    if (threadIdx.x < NCAP) {
      const int i = threadIdx.x;
      int64_t st0 = 0, d = 0;
      if (i < n && root_ok) row_range(rowptr, nodes[i], st0, d);
      rstart[i] = st0;
      rdeg[i] = (int32_t)d;
      chunks = row_chunks(d);
    }
    for (int i = threadIdx.x + kThreads; i < NCAP; i += kThreads) {  // NCAP > kThreads
      int64_t st0 = 0, d = 0;
      if (i < n && root_ok) row_range(rowptr, nodes[i], st0, d);
      rstart[i] = st0;
      rdeg[i] = (int32_t)d;
    }
    // chunk prefix over the rows (rows beyond kThreads are folded in serially)
    {
      int32_t tot;
      const int32_t pre = block_excl_scan(chunks, &tot, wsum);
      if (threadIdx.x < NCAP) cpre[threadIdx.x] = pre;
      __syncthreads();
      if (threadIdx.x == 0) {
        int32_t run = tot;
        for (int i = kThreads; i < NCAP; ++i) {
          cpre[i] = run;
          run += row_chunks(rdeg[i]);
        }
        cpre[NCAP] = run;
      }
      // rank of each node by global id -> ord[rank] = index
      for (int j = threadIdx.x; j < n; j += kThreads) {
        const int32_t g = nodes[j];
        int32_t rk = 0;
        for (int m = 0; m < n; ++m) rk += nodes[m] < g ? 1 : 0;
        ord[rk] = j;
      }
      __syncthreads();
    }
    const int32_t C = cpre[NCAP];
    for (int32_t c0 = wave * kChunkBatch; c0 < C; c0 += kWaves * kChunkBatch) {
      // row of chunk c0 by binary search, later chunks walk forward
      int lo = 0, hi = NCAP;  // cpre[lo] <= c0 < cpre[hi]
      while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (cpre[mid] <= c0) lo = mid;
        else hi = mid;
      }
      int32_t val[kChunkBatch];
      int rowu[kChunkBatch];
      int row = lo;
#pragma unroll
      for (int u = 0; u < kChunkBatch; ++u) {
        const int32_t c = c0 + u;
        val[u] = -1;
        rowu[u] = -1;
        if (c < C) {
          while (cpre[row + 1] <= c) ++row;
          const int32_t o = (c - cpre[row]) * 64 + lane;
          rowu[u] = row;
          if (o < rdeg[row]) val[u] = col[rstart[row] + o];
        }
      }
#pragma unroll
      for (int u = 0; u < kChunkBatch; ++u) {
        if (val[u] < 0) continue;
        const uint32_t b = fslot(val[u]);
        if (!((filt[b >> 5] >> (b & 31)) & 1u)) continue;
        const int32_t j = h_find(nk, nv, HCAP, val[u]);
        if (j >= 0 && j != rowu[u]) {
          const int32_t i = rowu[u];
          atomicOr(&bits[i * W + (j >> 5)], 1u << (j & 31));
          atomicOr(&bits[j * W + (i >> 5)], 1u << (i & 31));
        }
      }
    }
    // pairs of hubs
    {
      __shared__ int32_t hubs[NCAP];
      static_assert(NCAP <= kThreads, "one hub flag per thread");
      const int32_t is_hub = (threadIdx.x < n && root_ok && rdeg[threadIdx.x] > hub_deg) ? 1 : 0;
      int32_t nh;
      const int32_t pos = block_excl_scan(is_hub, &nh, wsum);
      if (is_hub) hubs[pos] = threadIdx.x;
      __syncthreads();
      for (int32_t p = threadIdx.x; p < nh * nh; p += kThreads) {
        const int32_t a = p / nh, bq = p - a * nh;
        if (bq <= a) continue;
        const int32_t i = hubs[a], j = hubs[bq];
        const bool i_short = rdeg[i] <= rdeg[j];
        const int32_t srow = i_short ? i : j, key = nodes[i_short ? j : i];
        int64_t lo = rstart[srow];
        const int64_t end = lo + rdeg[srow];
        int64_t hi = end;
        while (lo < hi) {
          const int64_t mid = (lo + hi) >> 1;
          if (col[mid] < key) lo = mid + 1;
          else hi = mid;
        }
        if (lo < end && col[lo] == key) {
          atomicOr(&bits[i * W + (j >> 5)], 1u << (j & 31));
          atomicOr(&bits[j * W + (i >> 5)], 1u << (i & 31));
        }
      }
    }
    __syncthreads();
    for (int32_t i = threadIdx.x; i < n && root_ok; i += kThreads) {
      int32_t* out = gedge + (int64_t)i * (nmax - 1);
      int32_t cnt = 0;
      for (int q = 0; q < n; ++q) {
        const int j = ord[q];
        if ((bits[i * W + (j >> 5)] >> (j & 31)) & 1u) out[cnt++] = j;
      }
      grow[i] = cnt;
      if (i == 0) e_root += cnt;
      else e_other += cnt;
    }
  } else {
    // induced edges: scan each node's CSR row, keep the neighbours in the set
    for (int32_t i = wave; i < n && root_ok; i += kWaves) {
      int64_t start, d;
      row_range(rowptr, nodes[i], start, d);
      int32_t cnt = 0;
      int32_t* out = gedge + (int64_t)i * (nmax - 1);
      for (int64_t c0 = 0; c0 < d; c0 += 64) {
        int32_t j = -1;
        if (c0 + lane < d) j = h_find(nk, nv, HCAP, col[start + c0 + lane]);
        const uint64_t m = ballot(j >= 0);
        const int32_t pre = __popcll(m & ((1ull << lane) - 1ull));
        // a simple graph has at most n - 1 matches per row; anything more is
        // malformed input and is dropped (flagged) rather than written
        if (j >= 0 && cnt + pre < nmax - 1) out[cnt + pre] = j;
        cnt += __popcll(m);
      }
      if (cnt > nmax - 1) {
        if (lane == 0) set_device_error(err, GNN_DEVERR_CAPACITY);
        cnt = nmax - 1;
      }
      if (lane == 0) {
        grow[i] = cnt;
        if (i == 0) e_root += cnt;
        else e_other += cnt;
      }
    }
  }
  if (!root_ok && threadIdx.x == 0) grow[0] = 0;
  // per-root totals
  int32_t t1, t2;
  block_excl_scan(e_root, &t1, wsum);
  block_excl_scan(e_other, &t2, wsum);
  if (threadIdx.x == 0) {
    int32_t* pr = stg.per_root + 4 * (int64_t)r;
    pr[0] = n;
    pr[1] = t1;
    pr[2] = t2;
    pr[3] = 0;
  }
}

// Exclusive prefix sums over roots of (other nodes, root-row edges, other-row
// edges) -> per_root_off [B x 4]; writes comp_ptr, the block counts and the
// readout counts.
__global__ void __launch_bounds__(1024)
shadow_scan_kernel(const int32_t* __restrict__ per_root, int32_t B, int32_t* __restrict__ off,
                   int32_t* __restrict__ comp_ptr, int32_t* counts, int32_t* readout_counts,
                   int32_t* indptr) {
  __shared__ int32_t wsum[3][16];
  __shared__ int32_t carry[3];
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  if (threadIdx.x < 3) carry[threadIdx.x] = 0;
  __syncthreads();
  for (int32_t c0 = 0; c0 < B; c0 += 1024) {
    const int32_t r = c0 + threadIdx.x;
    int32_t x[3] = {0, 0, 0};
    if (r < B) {
      x[0] = per_root[4 * r] - 1;
      x[1] = per_root[4 * r + 1];
      x[2] = per_root[4 * r + 2];
    }
    int32_t inc[3];
#pragma unroll
    for (int q = 0; q < 3; ++q) {
      inc[q] = wave_inclusive_scan(x[q]);
      if (lane == 63) wsum[q][wid] = inc[q];
    }
    __syncthreads();
    int32_t o[3], tot[3];
#pragma unroll
    for (int q = 0; q < 3; ++q) {
      o[q] = carry[q];
      tot[q] = 0;
      for (int w = 0; w < 16; ++w) {
        o[q] += (w < wid) ? wsum[q][w] : 0;
        tot[q] += wsum[q][w];
      }
      o[q] += inc[q] - x[q];
    }
    if (r < B) {
      off[4 * r] = o[0];
      off[4 * r + 1] = o[1];
      off[4 * r + 2] = o[2];
      off[4 * r + 3] = 0;
      comp_ptr[r] = B + o[0];
    }
    __syncthreads();
    if (threadIdx.x < 3) carry[threadIdx.x] += tot[threadIdx.x];
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    const int32_t total = B + carry[0];
    const int32_t e_total = carry[1] + carry[2];
    off[4 * B] = carry[0];
    off[4 * B + 1] = carry[1];
    off[4 * B + 2] = carry[2];
    off[4 * B + 3] = 0;
    comp_ptr[B] = total;
    counts[0] = total;
    counts[1] = total;
    counts[2] = e_total;
    counts[3] = 0;
    readout_counts[0] = B;
    readout_counts[1] = total;
    readout_counts[2] = carry[1];
    readout_counts[3] = 0;
    indptr[total] = e_total;
  }
}

// One workgroup per root: final local ids, rows, indices, src_nodes, src_occ.
__global__ void __launch_bounds__(kThreads)
shadow_emit_kernel(int32_t B, int32_t nmax, ShadowStage stg, const int32_t* __restrict__ off,
                   const int32_t* counts, int32_t* __restrict__ indptr,
                   int32_t* __restrict__ indices, int32_t* __restrict__ src_nodes,
                   int32_t* __restrict__ src_occ) {
  __shared__ int32_t wsum[kWaves];
  const int r = blockIdx.x;
  if (r >= B) return;
  const int32_t* pr = stg.per_root + 4 * (int64_t)r;
  const int32_t n = pr[0];
  const int32_t comp_base = B + off[4 * r];  // local id of component index 1
  const int32_t* gnodes = stg.nodes + (int64_t)r * nmax;
  const int32_t* grow = stg.rowcnt + (int64_t)r * nmax;
  const int32_t* gedge = stg.edges + (int64_t)r * nmax * (nmax - 1);
  auto local_of = [&](int32_t j) { return j == 0 ? r : comp_base + j - 1; };
  // row starts: the root row in the root segment; the others after every
  // root row (the root-row edge total is the scan's readout count)
  const int32_t root_start = off[4 * r + 1];
  const int32_t other_base = off[4 * (int64_t)B + 1] + off[4 * r + 2];
  // exclusive scan of the other rows' counts (rows 1..n-1), chunked
  int32_t run = 0;
  for (int32_t c0 = 1; c0 < n; c0 += kThreads) {
    const int32_t j = c0 + threadIdx.x;
    const int32_t x = j < n ? grow[j] : 0;
    int32_t tot;
    const int32_t pre = block_excl_scan(x, &tot, wsum);
    if (j < n) {
      const int32_t u = local_of(j);
      indptr[u] = other_base + run + pre;
      src_nodes[u] = gnodes[j];
      src_occ[u] = x + 1;
      const int32_t* ge = gedge + (int64_t)j * (nmax - 1);
      int32_t* oi = indices + other_base + run + pre;
      for (int32_t e = 0; e < x; ++e) oi[e] = local_of(ge[e]);
    }
    run += tot;
    __syncthreads();
  }
  // the root row
  if (threadIdx.x == 0) {
    indptr[r] = root_start;
    src_nodes[r] = gnodes[0];
    src_occ[r] = grow[0] + 1;
  }
  const int32_t x0 = grow[0];
  for (int32_t e = threadIdx.x; e < x0; e += kThreads) indices[root_start + e] = local_of(gedge[e]);
}

}  // namespace

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------
struct ShadowScratch {
  ShadowStage stg;
  int32_t* off;  // [(B + 1) x 4]
  size_t bytes;
};

static int shadow_plan(int32_t B, int32_t fanout, int32_t hops, void* ws, size_t ws_bytes,
                       ShadowScratch* s) {
  const int64_t nmax = shadow_max_nodes(fanout, hops);
  Carver c(ws, ws_bytes);
  s->stg.nodes = c.take<int32_t>((size_t)B * nmax);
  s->stg.rowcnt = c.take<int32_t>((size_t)B * nmax);
  s->stg.edges = c.take<int32_t>((size_t)std::max<int64_t>(1, (int64_t)B * nmax * (nmax - 1)));
  s->stg.per_root = c.take<int32_t>((size_t)std::max(1, B) * 4);
  s->off = c.take<int32_t>((size_t)(B + 1) * 4);
  s->bytes = c.off;
  return GNN_OK;
}

size_t shadow_scratch_bytes(int32_t B, int32_t fanout, int32_t hops) {
  ShadowScratch s;
  shadow_plan(B, fanout, hops, nullptr, 0, &s);
  return s.bytes;
}

template <typename RP>
static int shadow_launch(const gnn_csr* csr, const RP* rowptr, const int32_t* roots, int32_t B,
                         int32_t fanout, int32_t hops, uint64_t rng_key, gnn_block* sub,
                         int32_t* comp_ptr, int32_t* readout_counts, ShadowScratch& sc,
                         hipStream_t st) {
  const int64_t nmax = shadow_max_nodes(fanout, hops);
  int64_t cand_max = 1;
  for (int h = 0; h < hops; ++h) cand_max *= fanout;  // frontier x fanout at the last hop
  const int64_t need = std::max(nmax, cand_max);
  int* err = device_error_word();
  if (!err) return fail(GNN_EHIP, "device error word unavailable");
  if (need > 2048)
    return fail(GNN_EINVAL, "gnn_sample_shadow: %lld nodes per root exceed 2048", (long long)need);
  if (B > 0) {
    const int32_t hub = csr->hub_degree > 0 ? csr->hub_degree : kHubDegree;
    if (need <= 128)
      launch("shadow_build", shadow_build_kernel<128, RP>, B, kThreads, 0, st, rowptr, csr->col,
             csr->num_nodes, roots, B, fanout, hops, rng_key, (int32_t)nmax, sc.stg, err, hub);
    else if (need <= 512)
      launch("shadow_build", shadow_build_kernel<512, RP>, B, kThreads, 0, st, rowptr, csr->col,
             csr->num_nodes, roots, B, fanout, hops, rng_key, (int32_t)nmax, sc.stg, err, hub);
    else
      launch("shadow_build", shadow_build_kernel<2048, RP>, B, kThreads, 0, st, rowptr, csr->col,
             csr->num_nodes, roots, B, fanout, hops, rng_key, (int32_t)nmax, sc.stg, err, hub);
  }
  {
    launch("shadow_scan", shadow_scan_kernel, 1, 1024, 0, st, sc.stg.per_root, B, sc.off, comp_ptr,
           sub->counts, readout_counts, sub->indptr);
  }
  if (B > 0) {
    launch("shadow_emit", shadow_emit_kernel, B, kThreads, 0, st, B, (int32_t)nmax, sc.stg, sc.off,
           sub->counts, sub->indptr, sub->indices, sub->src_nodes, sub->src_occ);
  }
  GNN_LAUNCH_CHECK("gnn_sample_shadow");
  return GNN_OK;
}

int sample_shadow_impl(const gnn_csr* csr, const int32_t* roots, int32_t B, int32_t fanout,
                       int32_t hops, uint64_t rng_key, gnn_block* sub, int32_t* comp_ptr,
                       int32_t* readout_counts, void* ws, size_t ws_bytes, hipStream_t st) {
  ShadowScratch sc;
  shadow_plan(B, fanout, hops, ws, ws_bytes, &sc);
  if (sc.bytes > ws_bytes) return fail(GNN_EWORKSPACE, "gnn_sample_shadow: workspace too small");
  if (csr->rowptr_bits == 64)
    return shadow_launch(csr, static_cast<const int64_t*>(csr->rowptr), roots, B, fanout, hops,
                         rng_key, sub, comp_ptr, readout_counts, sc, st);
  return shadow_launch(csr, static_cast<const int32_t*>(csr->rowptr), roots, B, fanout, hops,
                       rng_key, sub, comp_ptr, readout_counts, sc, st);
}

int shadow_caps(int32_t B, int32_t fanout, int32_t hops, int32_t* cap_nodes, int64_t* cap_edges) {
  if (B < 0 || fanout < 1 || fanout > GNN_MAX_FANOUT || hops < 1 || hops > 3)
    return fail(GNN_EINVAL, "shadow: B >= 0, fanout in [1, 64], hops in [1, 3]");
  const int64_t nmax = shadow_max_nodes(fanout, hops);
  if (nmax > 2048) return fail(GNN_EINVAL, "shadow: %lld nodes per root exceed 2048", (long long)nmax);
  const int64_t nodes = (int64_t)B * nmax, edges = nodes * (nmax - 1);
  if (nodes > INT32_MAX || edges > INT32_MAX) return fail(GNN_EINVAL, "shadow: batch too large");
  *cap_nodes = (int32_t)nodes;
  *cap_edges = edges;
  return GNN_OK;
}

}  // namespace gnn

extern "C" {

int gnn_shadow_caps(int32_t B, int32_t fanout, int32_t hops, int32_t* cap_nodes, int64_t* cap_edges) {
  using namespace gnn;
  if (!cap_nodes || !cap_edges) return fail(GNN_EINVAL, "gnn_shadow_caps: null pointer");
  return shadow_caps(B, fanout, hops, cap_nodes, cap_edges);
}

size_t gnn_shadow_workspace_bytes(int32_t B, int32_t fanout, int32_t hops) {
  int32_t cn;
  int64_t ce;
  if (gnn::shadow_caps(B, fanout, hops, &cn, &ce) != GNN_OK) return 0;
  return gnn::shadow_scratch_bytes(B, fanout, hops);
}

int gnn_sample_shadow(const gnn_csr* csr, const int32_t* roots, int32_t B, int32_t fanout,
                      int32_t hops, uint64_t rng_key, gnn_block* sub, int32_t* comp_ptr,
                      int32_t* readout_counts, void* ws, size_t ws_bytes, void* stream) {
  using namespace gnn;
  if (!csr || !sub || !comp_ptr || !readout_counts || !ws || (B > 0 && !roots))
    return fail(GNN_EINVAL, "gnn_sample_shadow: null pointer");
  if (!csr->rowptr || !csr->col || (csr->rowptr_bits != 32 && csr->rowptr_bits != 64) ||
      csr->num_nodes < 0 || csr->num_nodes > INT32_MAX)
    return fail(GNN_EINVAL, "gnn_sample_shadow: bad CSR");
  if (int rc = check_csr_options(csr, "gnn_sample_shadow")) return rc;
  int32_t cn;
  int64_t ce;
  if (int rc = shadow_caps(B, fanout, hops, &cn, &ce)) return rc;
  if (!sub->indptr || !sub->indices || !sub->src_nodes || !sub->src_occ || !sub->counts)
    return fail(GNN_EINVAL, "gnn_sample_shadow: null block array");
  if (sub->cap_dst < cn || sub->cap_src < cn || sub->cap_edges < ce)
    return fail(GNN_EWORKSPACE, "gnn_sample_shadow: block capacities below gnn_shadow_caps");
  return sample_shadow_impl(csr, roots, B, fanout, hops, rng_key, sub, comp_ptr, readout_counts, ws,
                            ws_bytes, as_stream(stream));
}

}  // extern "C"
