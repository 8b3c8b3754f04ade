// GPU feature caching of a host-resident feature table (paper section 3, GPU
// Feature Caching): rows are fetched from a table the GPU reads in place over
// the host link (zero-copy), and a least-recently-used set of rows is kept in
// HBM, so that frequently needed rows cross the link once.
//
// The cache is set-associative (as HugeCTR's, which the paper adopts): node v
// lives in set fmix32(v) mod S, one of W ways, where fmix32 is MurmurHash3's
// 32-bit finaliser.  Recency is counted in fetch calls: call t stamps every
// entry it reads with t.  One call is four launches:
//   lookup  one lane group per requested row: compare the set's W keys, copy
//           the row from the cache (hit, re-stamped) or from host memory
//           (miss, counted per set; a set's first miss of the call appends
//           the set to the call's list of touched sets);
//   scan    each workgroup scans a chunk of the touched sets' miss counts and
//           reserves the chunk's slices of the miss list with one atomic
//           (offsets and cursors of those sets; where a set's slice lies does
//           not matter, only that its misses are contiguous);
//   place   each miss into its set's slice of a list; the call's header
//           words are reset and the call counter advances;
//   insert  one wave per touched set: its entries not read by this call are
//           replaced oldest stamp first (never used first, ties: lower way)
//           by the set's misses in request order, whose rows are copied from
//           the output just written (HBM to HBM); the set's miss count is
//           cleared for the next call.
// The work after the lookup follows the misses, not the number of sets, so a
// cache of millions of sets costs no more per call than a small one.
// Every choice is deterministic, so the cache's contents after any sequence
// of calls are reproducible.
#include <climits>

#include "internal.hpp"
#include "wave.hpp"

namespace gnn {

namespace {

constexpr int kThreads = 256;
constexpr int kMaxWays = 64;

struct CacheHeader {
  uint32_t calls;
  int32_t touched;    // sets appended to the touched list by this call's lookups
  int32_t list_next;  // the scan's next free position of the miss list
  uint32_t pad[61];
};

// Views of the caller's cache memory (layout fixed by carve_cache).
struct CacheView {
  CacheHeader* hdr;
  int32_t* keys;     // [S * W], -1 = empty
  uint32_t* stamps;  // [S * W], 0 = never used
  int32_t* miss_cnt; // [S], zero between calls
  uint4* rows;       // [S * W] rows of cpr 16-byte chunks
  int32_t S, W, cpr;
};

size_t carve_cache(Carver& c, int32_t S, int32_t W, int32_t cpr, CacheView* v) {
  v->hdr = c.take<CacheHeader>(1);
  v->keys = c.take<int32_t>((size_t)S * W);
  v->stamps = c.take<uint32_t>((size_t)S * W);
  v->miss_cnt = c.take<int32_t>((size_t)S);
  v->rows = c.take<uint4>((size_t)S * W * cpr);
  v->S = S;
  v->W = W;
  v->cpr = cpr;
  return c.off;
}

// Per-call scratch (only the entries of touched sets are written and read).
struct CallScratch {
  int32_t* off;       // [S]: first list position of a touched set's misses
  int32_t* cur;       // [S]: its placement cursor
  int32_t* miss_set;  // [cap]: set of a missed request, or -1
  int32_t* list;      // [cap]: request positions grouped by set
  int32_t* touched;   // [cap]: the sets with misses, in arrival order
  int32_t* n_touched; // [1]: their number (copied from the header by the scan)
};

size_t carve_call(Carver& c, int32_t S, int32_t cap, CallScratch* s) {
  s->off = c.take<int32_t>((size_t)S);
  s->cur = c.take<int32_t>((size_t)S);
  s->miss_set = c.take<int32_t>((size_t)std::max(1, cap));
  s->list = c.take<int32_t>((size_t)std::max(1, cap));
  s->touched = c.take<int32_t>((size_t)std::max(1, cap));
  s->n_touched = c.take<int32_t>(1);
  return c.off;
}

__device__ __forceinline__ uint32_t fmix32(uint32_t h) {
  h ^= h >> 16;
  h *= 0x85EBCA6Bu;
  h ^= h >> 13;
  h *= 0xC2B2AE35u;
  h ^= h >> 16;
  return h;
}

// Groups of G lanes, one requested row each (G >= the row's 16-byte chunks
// where possible, so a row is one load per lane).
// A set's first miss of the call goes to the workgroup's list in LDS; after
// each pass over its rows the workgroup appends the list to the call's
// touched list with one global atomic (one per set, from every workgroup,
// serialised on the one counter: about 60K of them per call on the 111M-node
// workload, 0.7 ms).  A pass adds at most one entry per lane group.
constexpr int kTouchedLds = kThreads;

template <int G>
__global__ void __launch_bounds__(kThreads)
lookup_kernel(CacheView cv, const uint4* __restrict__ X, int64_t n_rows, int64_t ld_x16,
              const int32_t* __restrict__ ids, const int32_t* n_ids, int32_t cap,
              uint4* __restrict__ out, int64_t ld_out16, int32_t* __restrict__ miss_set,
              int32_t* __restrict__ touched, unsigned long long* stats, int* err) {
  __shared__ int32_t red[2];
  __shared__ int32_t tl_n, tl_base;
  __shared__ int32_t tl[kTouchedLds];
  if (threadIdx.x < 2) red[threadIdx.x] = 0;
  if (threadIdx.x == 0) tl_n = 0;
  __syncthreads();
  // appends the workgroup's listed sets to the call's touched list (all threads)
  auto flush = [&]() {
    __syncthreads();
    const int32_t m = tl_n < kTouchedLds ? tl_n : kTouchedLds;
    if (threadIdx.x == 0 && m > 0) tl_base = atomicAdd(&cv.hdr->touched, m);
    __syncthreads();
    for (int32_t k = threadIdx.x; k < m; k += kThreads) touched[tl_base + k] = tl[k];
    __syncthreads();
    if (threadIdx.x == 0) tl_n = 0;
    __syncthreads();
  };
  int32_t n = *n_ids;
  if (n > cap) {
    if (blockIdx.x == 0 && threadIdx.x == 0) set_device_error(err, GNN_DEVERR_CAPACITY);
    n = cap;
  }
  const uint32_t t = cv.hdr->calls + 1;
  const int lane = lane_id(), r = lane & (G - 1);
  const int64_t group = ((int64_t)blockIdx.x * kThreads + threadIdx.x) / G;
  const int64_t groups = (int64_t)gridDim.x * (kThreads / G);
  int32_t hits = 0, misses = 0;
  // every thread runs the same number of passes (the flushes synchronise the
  // workgroup); a group past the last request idles through its pass
  const int64_t passes = (n + groups - 1) / groups;
  for (int64_t pass = 0; pass < passes; ++pass) {
    const int64_t i = group + pass * groups;
    if (i < n) {
      const int32_t id = ids[i];
      const bool valid = id >= 0 && (int64_t)id < n_rows;
      const int32_t s = valid ? (int32_t)(fmix32((uint32_t)id) % (uint32_t)cv.S) : 0;
      int32_t way = -1;
      if (valid)
        for (int w = r; w < cv.W; w += G)
          if (cv.keys[(int64_t)s * cv.W + w] == id) way = w;
#pragma unroll
      for (int d = G / 2; d >= 1; d >>= 1) way = max(way, __shfl_xor(way, d, WAVE));
      uint4* dst = out + i * ld_out16;
      if (way >= 0) {
        const uint4* src = cv.rows + ((int64_t)s * cv.W + way) * cv.cpr;
        for (int j = r; j < cv.cpr; j += G) dst[j] = src[j];
        if (r == 0) {
          cv.stamps[(int64_t)s * cv.W + way] = t;
          miss_set[i] = -1;
          ++hits;
        }
      } else {
        if (valid) {
          const uint4* src = X + (int64_t)id * ld_x16;
          for (int j = r; j < cv.cpr; j += G) dst[j] = src[j];
        } else {
          for (int j = r; j < cv.cpr; j += G) dst[j] = make_uint4(0, 0, 0, 0);
        }
        if (r == 0) {
          if (!valid) set_device_error(err, GNN_DEVERR_SEED_RANGE);
          else if (atomicAdd(&cv.miss_cnt[s], 1) == 0)  // the set's first miss of the call
            tl[atomicAdd(&tl_n, 1)] = s;
          miss_set[i] = valid ? s : -1;
          ++misses;
        }
      }
    }
    flush();
  }
  if (hits) atomicAdd(&red[0], hits);
  if (misses) atomicAdd(&red[1], misses);
  __syncthreads();
  if (threadIdx.x == 0 && (red[0] | red[1])) {
    atomicAdd(&stats[0], (unsigned long long)red[0]);
    atomicAdd(&stats[1], (unsigned long long)red[1]);
  }
}

// For the touched sets, off = cur = the first position of the set's slice of
// the miss list: each workgroup takes chunks of kThreads touched sets, scans
// their miss counts and reserves the chunk's range with one atomic (a single
// workgroup walking ~60K sets took ~0.25 ms per call on the 111M-node
// workload).  The touched count goes to the scratch.
__global__ void __launch_bounds__(kThreads)
scan_kernel(CacheView cv, CallScratch cs, int32_t cap) {
  __shared__ int32_t wsum[kThreads / 64];
  __shared__ int32_t s_base;
  int32_t nt = cv.hdr->touched;
  nt = nt > cap ? cap : nt;
  if (blockIdx.x == 0 && threadIdx.x == 0) *cs.n_touched = nt;
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  for (int64_t base = (int64_t)blockIdx.x * kThreads; base < nt; base += (int64_t)gridDim.x * kThreads) {
    const int64_t j = base + threadIdx.x;
    const int32_t set = j < nt ? cs.touched[j] : -1;
    const int32_t c = set >= 0 ? cv.miss_cnt[set] : 0;
    const int32_t inc = wave_inclusive_scan(c);
    if (lane == 63) wsum[wid] = inc;
    __syncthreads();
    int32_t before = 0, total = 0;
#pragma unroll
    for (int w = 0; w < kThreads / 64; ++w) {
      before += w < wid ? wsum[w] : 0;
      total += wsum[w];
    }
    if (threadIdx.x == 0) s_base = atomicAdd(&cv.hdr->list_next, total);
    __syncthreads();
    if (set >= 0) {
      cs.off[set] = s_base + before + inc - c;
      cs.cur[set] = s_base + before + inc - c;
    }
    __syncthreads();  // (wsum and s_base are rewritten by the next chunk)
  }
}

// Each miss into its set's slice; the first thread resets the call's header
// words (the next call's lookups append from 0) and advances the call counter
// (the insert launch stamps with it).
__global__ void __launch_bounds__(kThreads)
place_kernel(CacheView cv, const int32_t* n_ids, int32_t cap, CallScratch cs) {
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    cv.hdr->touched = 0;
    cv.hdr->list_next = 0;
    cv.hdr->calls = cv.hdr->calls + 1;
  }
  int32_t n = *n_ids;
  n = n > cap ? cap : n;
  for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * kThreads) {
    const int32_t s = cs.miss_set[i];
    if (s >= 0) cs.list[atomicAdd(&cs.cur[s], 1)] = (int32_t)i;
  }
}

__device__ __forceinline__ int32_t wave_min_i32(int32_t x) {
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) x = min(x, __shfl_xor(x, d, WAVE));
  return x;
}

// One wave per touched set.
__global__ void __launch_bounds__(kThreads)
insert_kernel(CacheView cv, CallScratch cs, const int32_t* __restrict__ ids,
              const uint4* __restrict__ out, int64_t ld_out16) {
  const int lane = lane_id();
  const uint32_t t = cv.hdr->calls;
  const int64_t wave = ((int64_t)blockIdx.x * kThreads + threadIdx.x) / WAVE;
  const int64_t waves = (int64_t)gridDim.x * (kThreads / WAVE);
  const int32_t nt = *cs.n_touched;
  for (int64_t q = wave; q < nt; q += waves) {
    const int32_t s = cs.touched[q];
    const int32_t lo = cs.off[s], m = cs.cur[s] - lo;  // the cursor ends past the set's misses
    if (lane == 0) cv.miss_cnt[s] = 0;                 // cleared for the next call
    const int64_t e0 = s * cv.W;
    const bool in = lane < cv.W;
    const uint32_t st = in ? cv.stamps[e0 + lane] : 0xFFFFFFFFu;
    const bool victim = in && st < t;
    // rank among the victims by (stamp, way)
    int32_t rank = 0;
    for (int u = 0; u < cv.W; ++u) {
      const uint32_t su = __shfl(st, u, WAVE);
      const bool vu = su < t;
      if (vu && (su < st || (su == st && u < lane))) ++rank;
    }
    const int32_t nv = __popcll(ballot(victim));
    const int32_t k = min(m, nv);
    int32_t prev = -1;
    for (int32_t j = 0; j < k; ++j) {
      // the j-th smallest request position among the set's misses
      int32_t best = INT_MAX;
      for (int32_t q = lane; q < m; q += WAVE) {
        const int32_t x = cs.list[lo + q];
        if (x > prev && x < best) best = x;
      }
      const int32_t sel = wave_min_i32(best);
      prev = sel;
      const uint64_t mask = ballot(victim && rank == j);
      const int w = __ffsll((unsigned long long)mask) - 1;
      if (lane == w) {
        cv.keys[e0 + w] = ids[sel];
        cv.stamps[e0 + w] = t;
      }
      const uint4* src = out + (int64_t)sel * ld_out16;
      uint4* dst = cv.rows + (e0 + w) * cv.cpr;
      for (int q = lane; q < cv.cpr; q += WAVE) dst[q] = src[q];
    }
  }
}

int check_cache(const gnn_feature_cache* c, int32_t* cpr, const char* who) {
  if (!c || !c->mem) return fail(GNN_EINVAL, "%s: null cache", who);
  if (c->num_sets < 1 || c->ways < 1 || c->ways > kMaxWays)
    return fail(GNN_EINVAL, "%s: num_sets >= 1 and ways in [1, %d]", who, kMaxWays);
  if (c->dtype != GNN_F32 && c->dtype != GNN_BF16) return fail(GNN_EINVAL, "%s: bad dtype", who);
  const int64_t es = c->dtype == GNN_F32 ? 4 : 2;
  if (c->width < 1 || ((int64_t)c->width * es) % 16)
    return fail(GNN_EINVAL, "%s: rows must be a positive multiple of 16 bytes", who);
  if ((int64_t)c->num_sets * c->ways > INT32_MAX / 2) return fail(GNN_EINVAL, "%s: cache too large", who);
  if (reinterpret_cast<uintptr_t>(c->mem) & 255) return fail(GNN_EINVAL, "%s: memory must be 256-byte aligned", who);
  *cpr = (int32_t)((int64_t)c->width * es / 16);
  return GNN_OK;
}

}  // namespace

}  // namespace gnn

extern "C" {

size_t gnn_feature_cache_bytes(int32_t num_sets, int32_t ways, int32_t width, int32_t dtype) {
  using namespace gnn;
  gnn_feature_cache c{num_sets, ways, width, dtype, reinterpret_cast<void*>(256)};
  int32_t cpr;
  if (check_cache(&c, &cpr, "gnn_feature_cache_bytes") != GNN_OK) return 0;
  Carver cv(nullptr, 0);
  CacheView v;
  return carve_cache(cv, num_sets, ways, cpr, &v);
}

int gnn_feature_cache_reset(const gnn_feature_cache* c, void* stream) {
  using namespace gnn;
  int32_t cpr;
  if (int rc = check_cache(c, &cpr, "gnn_feature_cache_reset")) return rc;
  Carver cv(c->mem, SIZE_MAX);
  CacheView v;
  carve_cache(cv, c->num_sets, c->ways, cpr, &v);
  const int64_t e = (int64_t)c->num_sets * c->ways;
  const FillRange fr[4] = {{v.hdr, (int64_t)(sizeof(CacheHeader) / 4), 0},
                           {v.keys, e, -1},
                           {v.stamps, e, 0},
                           {v.miss_cnt, c->num_sets, 0}};
  return launch_fill(fr, 4, as_stream(stream));
}

int gnn_feature_cache_views(const gnn_feature_cache* c, int32_t** keys, uint32_t** stamps,
                            void** rows) {
  using namespace gnn;
  int32_t cpr;
  if (int rc = check_cache(c, &cpr, "gnn_feature_cache_views")) return rc;
  Carver cv(c->mem, SIZE_MAX);
  CacheView v;
  carve_cache(cv, c->num_sets, c->ways, cpr, &v);
  if (keys) *keys = v.keys;
  if (stamps) *stamps = v.stamps;
  if (rows) *rows = v.rows;
  return GNN_OK;
}

size_t gnn_gather_cached_workspace_bytes(int32_t num_sets, int32_t cap) {
  using namespace gnn;
  if (num_sets < 1 || cap < 0) return 0;
  Carver c(nullptr, 0);
  CallScratch s;
  return carve_call(c, num_sets, cap, &s);
}

int gnn_gather_cached(const gnn_feature_cache* c, const void* X, int64_t n_rows, int64_t ld_x,
                      const int32_t* ids, const int32_t* n_ids, int32_t cap, void* out,
                      int64_t ld_out, uint64_t* stats, void* ws, size_t ws_bytes, void* stream) {
  using namespace gnn;
  const char* who = "gnn_gather_cached";
  int32_t cpr;
  if (int rc = check_cache(c, &cpr, who)) return rc;
  if (!X || !ids || !n_ids || !out || !stats || !ws) return fail(GNN_EINVAL, "%s: null pointer", who);
  if (cap < 0 || n_rows < 0) return fail(GNN_EINVAL, "%s: bad size", who);
  const int64_t es = c->dtype == GNN_F32 ? 4 : 2;
  if ((ld_x * es) % 16 || (ld_out * es) % 16 || ld_x < c->width || ld_out < c->width)
    return fail(GNN_EINVAL, "%s: strides must be 16-byte multiples >= the row width", who);
  if ((reinterpret_cast<uintptr_t>(X) | reinterpret_cast<uintptr_t>(out)) & 15)
    return fail(GNN_EINVAL, "%s: X and out must be 16-byte aligned", who);
  Carver cw(ws, ws_bytes);
  CallScratch cs;
  carve_call(cw, c->num_sets, cap, &cs);
  if (!cw.fits()) return fail(GNN_EWORKSPACE, "%s: workspace %zu < %zu bytes", who, ws_bytes, cw.off);
  if (cap == 0) return GNN_OK;
  Carver cc(c->mem, SIZE_MAX);
  CacheView v;
  carve_cache(cc, c->num_sets, c->ways, cpr, &v);
  int* err = device_error_word();
  if (!err) return fail(GNN_EHIP, "device error word unavailable");
  hipStream_t st = as_stream(stream);
  const int64_t ld_x16 = ld_x * es / 16, ld_out16 = ld_out * es / 16;
  auto outp = static_cast<uint4*>(out);
  const int G = cpr > 32 ? 64 : (cpr > 16 ? 32 : 16);
  const int64_t lblocks = std::min<int64_t>(8192, std::max<int64_t>(1, ceil_div((int64_t)cap * G, kThreads)));
  auto look = [&](auto kernel) {
    launch("cache_lookup", kernel, (unsigned)lblocks, kThreads, 0, st, v,
           static_cast<const uint4*>(X), n_rows, ld_x16, ids, n_ids, cap, outp, ld_out16,
           cs.miss_set, cs.touched, reinterpret_cast<unsigned long long*>(stats), err);
  };
  if (G == 16) look(lookup_kernel<16>);
  else if (G == 32) look(lookup_kernel<32>);
  else look(lookup_kernel<64>);
  GNN_LAUNCH_CHECK(who);
  const int64_t sblocks = std::min<int64_t>(512, std::max<int64_t>(1, ceil_div(cap, kThreads)));
  launch("cache_scan", scan_kernel, (unsigned)sblocks, kThreads, 0, st, v, cs, cap);
  GNN_LAUNCH_CHECK(who);
  const int64_t pblocks = std::min<int64_t>(2048, std::max<int64_t>(1, ceil_div(cap, kThreads)));
  launch("cache_place", place_kernel, (unsigned)pblocks, kThreads, 0, st, v, n_ids, cap, cs);
  GNN_LAUNCH_CHECK(who);
  const int64_t iblocks = std::min<int64_t>(
      8192, std::max<int64_t>(1, ceil_div(std::min<int64_t>(c->num_sets, cap), kThreads / WAVE)));
  launch("cache_insert", insert_kernel, (unsigned)iblocks, kThreads, 0, st, v, cs, ids,
         static_cast<const uint4*>(outp), ld_out16);
  GNN_LAUNCH_CHECK(who);
  return GNN_OK;
}

}  // extern "C"
