// Aggregation on a sampled block (Ahat H of paper section 2.1, eqs. (1)-(2)):
// a segmented reduction over the block's CSR rows, and its transpose (the
// scatter-add of the backward pass).
//
// Mapping: one wavefront per dst row.  The input rows can be addressed
// through the block's src node ids (the first layer then reads the feature
// table itself, with no separate gathered copy).  A row of H is split into
// 16-byte chunks; a group of LG lanes (LG = chunks per row rounded up to a
// power of two) holds one row.  The wave first loads its row's edge list,
// one edge per lane, then each group issues the 128-bit loads of several
// edges' rows before adding them, and the groups' partial sums are combined
// with cross-lane xor shuffles at the end of the row.
//
// Weights: GraphSAGE-mean w = 1/c_v (c_v sampled edges of v; 0 rows stay 0);
// GCN w = 1/sqrt(d_out(u) (c_v + 1)) with d_out(u) = src_occ[u] and one self
// edge per dst node; GIN-0 w = 1 on every sampled edge and on the self edge.
#include "internal.hpp"
#include "wave.hpp"

namespace gnn {

namespace {

constexpr int kThreads = 256;
// up to this many dst rows (one wave each) an aggregation keeps 16 rows in
// flight per wave; beyond, 8 (fewer registers, more resident waves)
constexpr int32_t kFewRows = 16384;

struct BlockDev {
  const int32_t* indptr;
  const int32_t* indices;
  const int32_t* occ;
  const int32_t* counts;
};

inline BlockDev dev_view(const gnn_block* b) {
  return BlockDev{b->indptr, b->indices, b->src_occ, b->counts};
}

// 16-byte chunk of a row as fp32 values (VEC = 4 for fp32, 8 for bf16)
template <int DT>
struct Chunk;

template <>
struct Chunk<GNN_F32> {
  static constexpr int VEC = 4;
  __device__ static inline void load(const void* base, int64_t idx16, float* v) {
    const float4 x = reinterpret_cast<const float4*>(base)[idx16];
    v[0] = x.x;
    v[1] = x.y;
    v[2] = x.z;
    v[3] = x.w;
  }
};

template <>
struct Chunk<GNN_BF16> {
  static constexpr int VEC = 8;
  __device__ static inline void load(const void* base, int64_t idx16, float* v) {
    const uint4 x = reinterpret_cast<const uint4*>(base)[idx16];
    const uint32_t w[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      v[2 * i] = __uint_as_float(w[i] << 16);
      v[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
    }
  }
};

// Rows of H: local row u is H row u, or, with a row map, H row rows[u] (row
// stride ld16 chunks; rows outside [0, n_rows) read as zeros, the sampler
// having flagged them already).
struct RowMap {
  const int32_t* rows;
  int64_t n_rows;
  int64_t ld16;
};

// H row of local row u (-1: reads as zeros)
__device__ __forceinline__ int32_t map_row(const RowMap& m, int32_t u) {
  if (!m.rows) return u;
  const int32_t r = m.rows[u];
  return r >= 0 && (int64_t)r < m.n_rows ? r : -1;
}

template <int N>
__device__ __forceinline__ void zero(float* x) {
#pragma unroll
  for (int i = 0; i < N; ++i) x[i] = 0.f;
}

// acc += sum over a row's c edges of w_e H[row_e] (this lane's chunk q), for
// one wave.  The edge list is taken 64 edges at a time, one per lane
// (edge(l, &row, &w) fills the H row, -1 for zeros, and the weight of edge
// l); each group of LG lanes then takes every G-th edge of the chunk and
// issues the row loads of U = EW / G edges before adding them in edge order
// (EW rows in flight per wave: 16 when the rows are few and the wave count
// small, 8 when the registers are better spent on more resident waves).
template <int DT, int LG, int EW, typename EdgeFn>
__device__ __forceinline__ void sum_rows(int32_t c, EdgeFn edge, const void* H, int64_t ld16,
                                         int q, bool active, float* acc) {
  using Ck = Chunk<DT>;
  constexpr int G = 64 / LG;
  constexpr int U = G >= EW ? 1 : EW / G;
  const int lane = lane_id();
  const int g = lane / LG;
  for (int32_t base = 0; base < c; base += 64) {
    const int32_t cc = c - base < 64 ? c - base : 64;
    int32_t my_row = -1;
    float my_w = 0.f;
    if (lane < cc) edge(base + lane, &my_row, &my_w);
    const int32_t kmax = (cc + G - 1) / G;
    for (int32_t k0 = 0; k0 < kmax; k0 += U) {
      float x[U][Ck::VEC];
      float wv[U];
#pragma unroll
      for (int k = 0; k < U; ++k) {
        const int32_t l = g + G * (k0 + k);
        const int32_t row = __shfl(my_row, l & 63, 64);
        const float w = __shfl(my_w, l & 63, 64);
        const bool ok = l < cc && row >= 0 && active;
        wv[k] = ok ? w : 0.f;
        if (ok) Ck::load(H, (int64_t)row * ld16 + q, x[k]);
        else zero<Ck::VEC>(x[k]);
      }
#pragma unroll
      for (int k = 0; k < U; ++k)
#pragma unroll
        for (int i = 0; i < Ck::VEC; ++i) acc[i] += wv[k] * x[k][i];
    }
  }
  // combine the groups
#pragma unroll
  for (int d = LG; d < 64; d <<= 1) {
#pragma unroll
    for (int i = 0; i < Ck::VEC; ++i) acc[i] += __shfl_xor(acc[i], d, 64);
  }
}

// X[v] = [H[v] | scale acc] (SAGE) or scale (acc + ws H[v]) (GCN, GIN), lane q's chunk
template <int DT, int KIND>
__device__ __forceinline__ void write_x(float* row, int32_t cpr, int q, const float* xs,
                                        float* acc, float scale, float ws) {
  using Ck = Chunk<DT>;
  if (KIND == GNN_SAGE_MEAN) {
    float4* so = reinterpret_cast<float4*>(row) + q * (Ck::VEC / 4);
#pragma unroll
    for (int i = 0; i < Ck::VEC / 4; ++i)
      so[i] = make_float4(xs[4 * i], xs[4 * i + 1], xs[4 * i + 2], xs[4 * i + 3]);
    row += cpr * Ck::VEC;  // the aggregate starts at column F
  } else {
#pragma unroll
    for (int i = 0; i < Ck::VEC; ++i) acc[i] += ws * xs[i];
  }
  float4* ao = reinterpret_cast<float4*>(row) + q * (Ck::VEC / 4);
#pragma unroll
  for (int i = 0; i < Ck::VEC / 4; ++i)
    ao[i] = make_float4(acc[4 * i] * scale, acc[4 * i + 1] * scale, acc[4 * i + 2] * scale,
                        acc[4 * i + 3] * scale);
}

template <int DT, int KIND, int LG, int EW>
__global__ void __launch_bounds__(kThreads)
aggregate_kernel(BlockDev b, const void* __restrict__ H, int32_t cpr, RowMap map,
                 float* __restrict__ out, int32_t out_ld, int32_t agg_blocks, FillPair fills) {
  if ((int32_t)blockIdx.x >= agg_blocks) {
    run_fills(fills, blockIdx.x - agg_blocks, gridDim.x - agg_blocks, kThreads);
    return;
  }
  using C = Chunk<DT>;
  const int lane = lane_id();
  const int q = lane % LG;
  const int64_t v = ((int64_t)blockIdx.x * kThreads + threadIdx.x) >> 6;
  if (v >= b.counts[0]) return;
  const int32_t e0 = b.indptr[v], e1 = b.indptr[v + 1];
  const int32_t c = e1 - e0;
  const bool active = q < cpr;
  const int64_t ld16 = map.rows ? map.ld16 : cpr;
  // the dst node v is also local src row v; its row is loaded up front
  const int32_t rs = map_row(map, (int32_t)v);
  float xs[C::VEC];
  if (active && rs >= 0) C::load(H, (int64_t)rs * ld16 + q, xs);
  else zero<C::VEC>(xs);
  float acc[C::VEC];
  zero<C::VEC>(acc);
  auto edge = [&](int32_t l, int32_t* row, float* w) {
    const int32_t u = b.indices[e0 + l];
    *row = map_row(map, u);
    *w = KIND == GNN_GCN ? rsqrtf((float)b.occ[u]) : 1.f;
  };
  sum_rows<DT, LG, EW>(c, edge, H, ld16, q, active, acc);
  if (lane >= LG || !active) return;
  float scale, ws = 0.f;
  if (KIND == GNN_SAGE_MEAN) {
    scale = c > 0 ? 1.f / (float)c : 0.f;
  } else if (KIND == GNN_GIN) {
    ws = 1.f;
    scale = 1.f;
  } else {
    ws = rsqrtf((float)b.occ[v]);  // self edge
    scale = rsqrtf((float)(c + 1));
  }
  write_x<DT, KIND>(out + v * (int64_t)out_ld, cpr, q, xs, acc, scale, ws);
}

// GraphSAGE-mean aggregation of the last sampled hop straight from its
// padded picks (slot (v, r), r < kcount[v], holds the global id of a sampled
// neighbour of dst v), reading rows of the feature table X: the same sums, in
// the same order, as over the compacted block, but without waiting for the
// compaction, which blocks past agg_blocks run meanwhile.  A pick with an
// invalid id (device error raised by the sampler) reads as local row 0, as in
// the compacted block.
template <int DT, int LG, int EW>
__global__ void __launch_bounds__(kThreads)
aggregate_picks_kernel(SampleTail tail, const int32_t* __restrict__ src_nodes,
                       const void* __restrict__ H, int32_t cpr, int64_t n_rows, int64_t ld16,
                       float* __restrict__ out, int32_t out_ld, int32_t agg_blocks) {
  if ((int32_t)blockIdx.x >= agg_blocks) {
    finish_sampling(tail, blockIdx.x - agg_blocks, gridDim.x - agg_blocks, kThreads);
    return;
  }
  using C = Chunk<DT>;
  const IndexJob& j = tail.job;
  const int lane = lane_id();
  const int q = lane % LG;
  const int64_t v = ((int64_t)blockIdx.x * kThreads + threadIdx.x) >> 6;
  if (v >= j.counts[0]) return;
  const int32_t c = j.kcount[v];
  const int32_t* picks = j.nbr_pad + v * (int64_t)j.fanout;
  const bool active = q < cpr;
  auto valid = [&](int32_t r) { return r >= 0 && (int64_t)r < n_rows; };
  const int32_t sv = src_nodes[v];
  float xs[C::VEC];
  if (active && valid(sv)) C::load(H, (int64_t)sv * ld16 + q, xs);
  else zero<C::VEC>(xs);
  // global row of local src 0 (the first dst node): invalid picks read it
  const int32_t row0 = src_nodes[0];
  float acc[C::VEC];
  zero<C::VEC>(acc);
  auto edge = [&](int32_t l, int32_t* row, float* w) {
    const int32_t key = picks[l];
    const int32_t r = valid(key) ? key : row0;
    *row = valid(r) ? r : -1;
    *w = 1.f;
  };
  sum_rows<DT, LG, EW>(c, edge, H, ld16, q, active, acc);
  if (lane >= LG || !active) return;
  write_x<DT, GNN_SAGE_MEAN>(out + v * (int64_t)out_ld, cpr, q, xs, acc, c > 0 ? 1.f / (float)c : 0.f,
                             0.f);
}

// dH[u] += w_e dAgg[v] for every edge (v, u) (+ GCN / GIN self edge), fp32 atomics.
// A group of LG lanes owns one edge; lane q handles features q, q + LG, ...,
// so every atomic instruction covers LG consecutive floats of one row.
template <int KIND, int LG>
__global__ void __launch_bounds__(kThreads)
scatter_kernel(BlockDev b, const float* __restrict__ dAgg, float* dH, int32_t F) {
  constexpr int G = 64 / LG;
  constexpr int NV = LG == 64 ? 4 : 1;  // F <= 256
  const int lane = lane_id();
  const int g = lane / LG, q = lane % LG;
  const int64_t v = ((int64_t)blockIdx.x * kThreads + threadIdx.x) >> 6;
  if (v >= b.counts[0]) return;
  const int32_t e0 = b.indptr[v], e1 = b.indptr[v + 1];
  const int32_t c = e1 - e0;
  float d[NV];
#pragma unroll
  for (int j = 0; j < NV; ++j) {
    const int f = q + j * LG;
    d[j] = f < F ? dAgg[v * (int64_t)F + f] : 0.f;
  }
  float rs;
  if (KIND == GNN_SAGE_MEAN) {
    if (c == 0) return;
    rs = 1.f / (float)c;
  } else {
    rs = KIND == GNN_GIN ? 1.f : rsqrtf((float)(c + 1));
    if (g == 0) {
      const float w = KIND == GNN_GIN ? 1.f : rs * rsqrtf((float)b.occ[v]);
      float* o = dH + v * (int64_t)F;
#pragma unroll
      for (int j = 0; j < NV; ++j) {
        const int f = q + j * LG;
        if (f < F) unsafeAtomicAdd(o + f, w * d[j]);
      }
    }
  }
  // the edge list 64 at a time, one edge (src row, weight) per lane; the
  // atomics then issue back to back
  for (int32_t base = 0; base < c; base += 64) {
    const int32_t cc = c - base < 64 ? c - base : 64;
    int32_t my_u = 0;
    float my_w = 0.f;
    if (lane < cc) {
      my_u = b.indices[e0 + base + lane];
      my_w = KIND == GNN_GCN ? rs * rsqrtf((float)b.occ[my_u]) : rs;
    }
    for (int32_t l0 = 0; l0 < cc; l0 += G) {
      const int32_t l = l0 + g;
      const int32_t u = __shfl(my_u, l & 63, 64);
      const float w = __shfl(my_w, l & 63, 64);
      if (l < cc) {
        float* o = dH + (int64_t)u * F;
#pragma unroll
        for (int j = 0; j < NV; ++j) {
          const int f = q + j * LG;
          if (f < F) unsafeAtomicAdd(o + f, w * d[j]);
        }
      }
    }
  }
}

// The same backward as a gather over the block's transpose: one wave per src
// row u < n_src, dH[u] = sum over u's edges (v, u) of w_e dAgg[v] (+ GCN / GIN
// self edge for a dst u), written once (no atomics, no zeroing).  SAGE: rows u <
// n_dst already hold the self path (the dX product wrote them) and are added
// to; the other rows are overwritten.
template <int KIND, int LG, int EW>
__global__ void __launch_bounds__(kThreads)
scatter_t_kernel(BlockDev b, const int32_t* __restrict__ t_ptr, const int32_t* __restrict__ t_dst,
                 const float* __restrict__ dAgg, float* __restrict__ dH, int32_t F) {
  using C = Chunk<GNN_F32>;
  const int lane = lane_id();
  const int q = lane % LG;
  const int64_t u = ((int64_t)blockIdx.x * kThreads + threadIdx.x) >> 6;
  if (u >= b.counts[1]) return;
  const int32_t n_dst = b.counts[0];
  const int32_t cpr = F / 4;
  const bool active = q < cpr;
  const int32_t l0 = t_ptr[u], c = t_ptr[u + 1] - l0;
  float ru = 1.f;
  if (KIND == GNN_GCN) ru = rsqrtf((float)b.occ[u]);
  float acc[C::VEC];
  zero<C::VEC>(acc);
  auto edge = [&](int32_t l, int32_t* row, float* w) {
    const int32_t v = t_dst[l0 + l];
    const int32_t cv = b.indptr[v + 1] - b.indptr[v];
    *row = v;
    *w = KIND == GNN_GCN ? ru * rsqrtf((float)(cv + 1)) : (KIND == GNN_GIN ? 1.f : 1.f / (float)cv);
  };
  sum_rows<GNN_F32, LG, EW>(c, edge, dAgg, cpr, q, active, acc);
  if (lane >= LG || !active) return;
  float4* o = reinterpret_cast<float4*>(dH + u * (int64_t)F) + q;
  if (u < n_dst) {
    if (KIND != GNN_SAGE_MEAN) {
      // self edge of dst u
      const float ws = KIND == GNN_GIN ? 1.f : ru * rsqrtf((float)(b.indptr[u + 1] - b.indptr[u] + 1));
      const float4 d = reinterpret_cast<const float4*>(dAgg + u * (int64_t)F)[q];
      acc[0] += ws * d.x;
      acc[1] += ws * d.y;
      acc[2] += ws * d.z;
      acc[3] += ws * d.w;
    } else {
      const float4 s = *o;
      acc[0] += s.x;
      acc[1] += s.y;
      acc[2] += s.z;
      acc[3] += s.w;
    }
  }
  *o = make_float4(acc[0], acc[1], acc[2], acc[3]);
}

__global__ void __launch_bounds__(kThreads)
relu_mask_kernel(const int32_t* rows_dev, int32_t cap, const float4* __restrict__ h,
                 float4* __restrict__ x, int32_t c4) {
  int32_t rows = *rows_dev;
  rows = rows > cap ? cap : rows;
  const int64_t n = (int64_t)rows * c4;
  for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * kThreads) {
    const float4 m = h[i];
    float4 y = x[i];
    y.x = m.x > 0.f ? y.x : 0.f;
    y.y = m.y > 0.f ? y.y : 0.f;
    y.z = m.z > 0.f ? y.z : 0.f;
    y.w = m.w > 0.f ? y.w : 0.f;
    x[i] = y;
  }
}


inline int pow2_at_least(int x) {
  int p = 1;
  while (p < x) p <<= 1;
  return p;
}

template <int DT, int KIND>
int dispatch_aggregate(const gnn_block* blk, const void* H, int32_t F, const RowMap& map,
                       float* agg, int32_t out_ld, const FillPair& fills, hipStream_t st) {
  const int32_t es = DT == GNN_F32 ? 4 : 2;
  const int32_t cpr = F * es / 16;
  const int lg = pow2_at_least(cpr);
  const int64_t ablocks = std::max<int64_t>(1, ceil_div((int64_t)blk->cap_dst * 64, kThreads));
  const unsigned grid = (unsigned)(ablocks + fill_blocks(fills, kThreads));
  BlockDev b = dev_view(blk);
  auto go = [&](auto kernel) {
    launch("aggregate", kernel, grid, kThreads, 0, st, b, H, cpr, map, agg, out_ld,
           (int32_t)ablocks, fills);
  };
  // rows in flight per wave: more while the rows fit the resident waves
  const bool few = blk->cap_dst <= kFewRows;
#define GNN_AGG_CASE(N)                                                    \
  case N:                                                                  \
    if (few) go(aggregate_kernel<DT, KIND, N, 16>);                        \
    else go(aggregate_kernel<DT, KIND, N, 8>);                             \
    break;
  switch (lg) {
    GNN_AGG_CASE(1)
    GNN_AGG_CASE(2)
    GNN_AGG_CASE(4)
    GNN_AGG_CASE(8)
    GNN_AGG_CASE(16)
    GNN_AGG_CASE(32)
    GNN_AGG_CASE(64)
    default: return fail(GNN_EINVAL, "aggregate: feature row of %d chunks > 64", cpr);
  }
#undef GNN_AGG_CASE
  GNN_LAUNCH_CHECK("aggregate");
  return GNN_OK;
}

template <int DT>
int dispatch_aggregate_picks(const SampleTail& tail, int32_t cap_dst, const int32_t* src_nodes,
                             const void* H, int32_t F, int64_t n_rows, int64_t ld16, float* out,
                             int32_t out_ld, hipStream_t st) {
  const int32_t es = DT == GNN_F32 ? 4 : 2;
  const int32_t cpr = F * es / 16;
  const int lg = pow2_at_least(cpr);
  const int64_t ablocks = std::max<int64_t>(1, ceil_div((int64_t)cap_dst * 64, kThreads));
  const int64_t slots = (int64_t)cap_dst * tail.job.fanout;
  const int64_t tblocks = std::min<int64_t>(1024, std::max<int64_t>(1, ceil_div(slots, kThreads * 4)));
  auto go = [&](auto kernel) {
    launch("aggregate", kernel, (unsigned)(ablocks + tblocks), kThreads, 0, st, tail, src_nodes, H,
           cpr, n_rows, ld16, out, out_ld, (int32_t)ablocks);
  };
  const bool few = cap_dst <= kFewRows;
#define GNN_AGG_CASE(N)                                      \
  case N:                                                    \
    if (few) go(aggregate_picks_kernel<DT, N, 16>);          \
    else go(aggregate_picks_kernel<DT, N, 8>);               \
    break;
  switch (lg) {
    GNN_AGG_CASE(1)
    GNN_AGG_CASE(2)
    GNN_AGG_CASE(4)
    GNN_AGG_CASE(8)
    GNN_AGG_CASE(16)
    GNN_AGG_CASE(32)
    GNN_AGG_CASE(64)
    default: return fail(GNN_EINVAL, "aggregate: feature row of %d chunks > 64", cpr);
  }
#undef GNN_AGG_CASE
  GNN_LAUNCH_CHECK("aggregate");
  return GNN_OK;
}

template <int KIND>
int dispatch_scatter(const gnn_block* blk, const float* dAgg, int32_t F, float* dH, hipStream_t st) {
  const int lg = F >= 64 ? 64 : pow2_at_least(F);
  const unsigned grid = (unsigned)std::max<int64_t>(1, ceil_div((int64_t)blk->cap_dst * 64, kThreads));
  BlockDev b = dev_view(blk);
  auto go = [&](auto kernel) { launch("scatter", kernel, grid, kThreads, 0, st, b, dAgg, dH, F); };
  switch (lg) {
    case 4: go(scatter_kernel<KIND, 4>); break;
    case 8: go(scatter_kernel<KIND, 8>); break;
    case 16: go(scatter_kernel<KIND, 16>); break;
    case 32: go(scatter_kernel<KIND, 32>); break;
    case 64: go(scatter_kernel<KIND, 64>); break;
    default: return fail(GNN_EINVAL, "scatter: feature width %d", F);
  }
  GNN_LAUNCH_CHECK("scatter");
  return GNN_OK;
}

}  // namespace

int launch_aggregate(const gnn_block* blk, int32_t kind, const void* H, int32_t dtype, int32_t F,
                     float* out, int32_t out_ld, hipStream_t st, const int32_t* rows,
                     int64_t n_rows, int64_t ld_h, const FillPair& fills) {
  if (blk->cap_dst == 0) {
    FillRange fr[2];
    int n = 0;
    for (int r = 0; r < 2; ++r)
      if (fills.n[r] > 0) fr[n++] = FillRange{fills.p[r], fills.n[r], fills.v[r]};
    return launch_fill(fr, n, st);
  }
  const int32_t es = dtype == GNN_F32 ? 4 : 2;
  if (rows && ((ld_h * es) % 16 || ld_h < F)) return fail(GNN_EINVAL, "aggregate: bad row stride");
  const RowMap map{rows, n_rows, rows ? ld_h * es / 16 : 0};
  if (dtype == GNN_F32) {
    if (kind == GNN_GCN) return dispatch_aggregate<GNN_F32, GNN_GCN>(blk, H, F, map, out, out_ld, fills, st);
    if (kind == GNN_GIN) return dispatch_aggregate<GNN_F32, GNN_GIN>(blk, H, F, map, out, out_ld, fills, st);
    return dispatch_aggregate<GNN_F32, GNN_SAGE_MEAN>(blk, H, F, map, out, out_ld, fills, st);
  }
  if (kind == GNN_GCN) return dispatch_aggregate<GNN_BF16, GNN_GCN>(blk, H, F, map, out, out_ld, fills, st);
  if (kind == GNN_GIN) return dispatch_aggregate<GNN_BF16, GNN_GIN>(blk, H, F, map, out, out_ld, fills, st);
  return dispatch_aggregate<GNN_BF16, GNN_SAGE_MEAN>(blk, H, F, map, out, out_ld, fills, st);
}

int launch_aggregate_picks(const SampleTail& tail, const gnn_block* blk, const void* H,
                           int32_t dtype, int32_t F, int64_t n_rows, int64_t ld_h, float* out,
                           int32_t out_ld, hipStream_t st) {
  const int32_t es = dtype == GNN_F32 ? 4 : 2;
  if ((ld_h * es) % 16 || ld_h < F) return fail(GNN_EINVAL, "aggregate: bad row stride");
  if (dtype == GNN_F32)
    return dispatch_aggregate_picks<GNN_F32>(tail, blk->cap_dst, blk->src_nodes, H, F, n_rows,
                                             ld_h * es / 16, out, out_ld, st);
  return dispatch_aggregate_picks<GNN_BF16>(tail, blk->cap_dst, blk->src_nodes, H, F, n_rows,
                                            ld_h * es / 16, out, out_ld, st);
}

int launch_scatter(const gnn_block* blk, int32_t kind, const float* dAgg, int32_t F, float* dH,
                   hipStream_t st) {
  if (blk->cap_dst == 0) return GNN_OK;
  if (kind == GNN_GCN) return dispatch_scatter<GNN_GCN>(blk, dAgg, F, dH, st);
  if (kind == GNN_GIN) return dispatch_scatter<GNN_GIN>(blk, dAgg, F, dH, st);
  return dispatch_scatter<GNN_SAGE_MEAN>(blk, dAgg, F, dH, st);
}

int launch_scatter_t(const gnn_block* blk, int32_t kind, const int32_t* t_ptr, const int32_t* t_dst,
                     const float* dAgg, int32_t F, float* dH, hipStream_t st) {
  if (blk->cap_src == 0) return GNN_OK;
  if (F % 4 || F > 256) return fail(GNN_EINVAL, "scatter: feature width %d", F);
  const int lg = pow2_at_least(F / 4);
  const unsigned grid = (unsigned)std::max<int64_t>(1, ceil_div((int64_t)blk->cap_src * 64, kThreads));
  BlockDev b = dev_view(blk);
  auto go = [&](auto kernel) { launch("scatter", kernel, grid, kThreads, 0, st, b, t_ptr, t_dst, dAgg, dH, F); };
#define GNN_ST_CASE(N)                                          \
  case N:                                                       \
    if (kind == GNN_GCN) go(scatter_t_kernel<GNN_GCN, N, 8>);   \
    else if (kind == GNN_GIN) go(scatter_t_kernel<GNN_GIN, N, 8>); \
    else go(scatter_t_kernel<GNN_SAGE_MEAN, N, 8>);             \
    break;
  switch (lg) {
    GNN_ST_CASE(1)
    GNN_ST_CASE(2)
    GNN_ST_CASE(4)
    GNN_ST_CASE(8)
    GNN_ST_CASE(16)
    GNN_ST_CASE(32)
    GNN_ST_CASE(64)
    default: return fail(GNN_EINVAL, "scatter: feature width %d", F);
  }
#undef GNN_ST_CASE
  GNN_LAUNCH_CHECK("scatter");
  return GNN_OK;
}

int launch_relu_mask(const gnn_block* blk, const float* h, int32_t F, float* x, hipStream_t st) {
  const int32_t c4 = F / 4;
  int64_t blocks = ceil_div((int64_t)blk->cap_src * c4, kThreads * 4);
  blocks = blocks < 1 ? 1 : (blocks > 4096 ? 4096 : blocks);
  launch("relu_mask", relu_mask_kernel, (unsigned)blocks, kThreads, 0, st, blk->counts + 1,
         blk->cap_src, reinterpret_cast<const float4*>(h), reinterpret_cast<float4*>(x), c4);
  GNN_LAUNCH_CHECK("relu mask");
  return GNN_OK;
}


}  // namespace gnn
