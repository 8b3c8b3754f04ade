// Aggregation on a sampled block (Ahat H of paper section 2.1, eqs. (1)-(2)):
// a segmented reduction over the block's CSR rows, and its transpose (the
// scatter-add of the backward pass).
//
// Mapping: one wavefront per dst row.  The input rows can be addressed
// through the block's src node ids (the first layer then reads the feature
// table itself, with no separate gathered copy).  A row of H is split into 16-byte
// chunks; a group of LG lanes (LG = chunks per row rounded up to a power of
// two) holds one row, so a wave works on 64 / LG edges at once, each lane
// issuing 128-bit loads.  The groups' partial sums are combined with
// cross-lane xor shuffles at the end of the row.
//
// Weights: GraphSAGE-mean w = 1/c_v (c_v sampled edges of v; 0 rows stay 0);
// GCN w = 1/sqrt(d_out(u) (c_v + 1)) with d_out(u) = src_occ[u] and one self
// edge per dst node.
#include "internal.hpp"
#include "wave.hpp"

namespace gnn {

namespace {

constexpr int kThreads = 256;

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

__device__ __forceinline__ int64_t row_chunk(const RowMap& m, int32_t cpr, int32_t u, bool* ok) {
  if (!m.rows) {
    *ok = true;
    return (int64_t)u * cpr;
  }
  const int32_t r = m.rows[u];
  *ok = r >= 0 && (int64_t)r < m.n_rows;
  return (*ok ? (int64_t)r : 0) * m.ld16;
}

template <int N>
__device__ __forceinline__ void zero(float* x) {
#pragma unroll
  for (int i = 0; i < N; ++i) x[i] = 0.f;
}

template <int DT, int KIND, int LG>
__global__ void __launch_bounds__(kThreads)
aggregate_kernel(BlockDev b, const void* __restrict__ H, int32_t cpr, RowMap map,
                 float* __restrict__ out, int32_t out_ld) {
  using C = Chunk<DT>;
  constexpr int G = 64 / LG;
  const int lane = lane_id();
  const int g = lane / LG, q = lane % LG;
  const int64_t v = ((int64_t)blockIdx.x * kThreads + threadIdx.x) >> 6;
  if (v >= b.counts[0]) return;
  const int32_t e0 = b.indptr[v], e1 = b.indptr[v + 1];
  const bool active = q < cpr;
  float acc[C::VEC];
#pragma unroll
  for (int i = 0; i < C::VEC; ++i) acc[i] = 0.f;
  int32_t e = e0 + g;
  // two edges per group in flight
  for (; e + G < e1; e += 2 * G) {
    const int32_t u0 = b.indices[e], u1 = b.indices[e + G];
    float x0[C::VEC], x1[C::VEC];
    bool ok0, ok1;
    const int64_t r0 = row_chunk(map, cpr, u0, &ok0), r1 = row_chunk(map, cpr, u1, &ok1);
    if (active) {
      C::load(H, r0 + q, x0);
      C::load(H, r1 + q, x1);
      if (!ok0) zero<C::VEC>(x0);
      if (!ok1) zero<C::VEC>(x1);
      float w0 = 1.f, w1 = 1.f;
      if (KIND == GNN_GCN) {
        w0 = rsqrtf((float)b.occ[u0]);
        w1 = rsqrtf((float)b.occ[u1]);
      }
#pragma unroll
      for (int i = 0; i < C::VEC; ++i) acc[i] += w0 * x0[i] + w1 * x1[i];
    }
  }
  if (e < e1 && active) {
    const int32_t u0 = b.indices[e];
    float x0[C::VEC];
    bool ok0;
    const int64_t r0 = row_chunk(map, cpr, u0, &ok0);
    C::load(H, r0 + q, x0);
    if (!ok0) zero<C::VEC>(x0);
    const float w0 = KIND == GNN_GCN ? rsqrtf((float)b.occ[u0]) : 1.f;
#pragma unroll
    for (int i = 0; i < C::VEC; ++i) acc[i] += w0 * x0[i];
  }
  // combine the groups
#pragma unroll
  for (int d = LG; d < 64; d <<= 1) {
#pragma unroll
    for (int i = 0; i < C::VEC; ++i) acc[i] += __shfl_xor(acc[i], d, 64);
  }
  if (g != 0 || !active) return;
  const int32_t c = e1 - e0;
  float* row = out + v * (int64_t)out_ld;
  float scale;
  // the dst node v is also local src row v
  bool oks;
  const int64_t rs = row_chunk(map, cpr, (int32_t)v, &oks);
  if (KIND == GNN_SAGE_MEAN) {
    scale = c > 0 ? 1.f / (float)c : 0.f;
    // self row (widened to fp32) next to the aggregate: X[v] = [H[v] | agg_v]
    float xs[C::VEC];
    C::load(H, rs + q, xs);
    if (!oks) zero<C::VEC>(xs);
    float4* so = reinterpret_cast<float4*>(row) + q * (C::VEC / 4);
#pragma unroll
    for (int i = 0; i < C::VEC / 4; ++i)
      so[i] = make_float4(xs[4 * i], xs[4 * i + 1], xs[4 * i + 2], xs[4 * i + 3]);
    row += cpr * C::VEC;  // the aggregate starts at column F
  } else {
    // self edge
    float xs[C::VEC];
    C::load(H, rs + q, xs);
    if (!oks) zero<C::VEC>(xs);
    const float ws = rsqrtf((float)b.occ[v]);
#pragma unroll
    for (int i = 0; i < C::VEC; ++i) acc[i] += ws * xs[i];
    scale = rsqrtf((float)(c + 1));
  }
  float4* ao = reinterpret_cast<float4*>(row) + q * (C::VEC / 4);
#pragma unroll
  for (int i = 0; i < C::VEC / 4; ++i)
    ao[i] = make_float4(acc[4 * i] * scale, acc[4 * i + 1] * scale, acc[4 * i + 2] * scale,
                        acc[4 * i + 3] * scale);
}

// GraphSAGE-mean aggregation of the last sampled hop straight from its
// padded picks (slot (v, r), r < kcount[v], holds the global id of a sampled
// neighbour of dst v), reading rows of the feature table X: the same sums, in
// the same order, as over the compacted block, but without waiting for the
// compaction, which blocks past agg_blocks run meanwhile.  A pick with an
// invalid id (device error raised by the sampler) reads as local row 0, as in
// the compacted block.
template <int DT, int LG>
__global__ void __launch_bounds__(kThreads)
aggregate_picks_kernel(SampleTail tail, const int32_t* __restrict__ src_nodes,
                       const void* __restrict__ H, int32_t cpr, int64_t n_rows, int64_t ld16,
                       float* __restrict__ out, int32_t out_ld, int32_t agg_blocks) {
  if ((int32_t)blockIdx.x >= agg_blocks) {
    finish_sampling(tail, blockIdx.x - agg_blocks, gridDim.x - agg_blocks, kThreads);
    return;
  }
  using C = Chunk<DT>;
  constexpr int G = 64 / LG;
  const IndexJob& j = tail.job;
  const int lane = lane_id();
  const int g = lane / LG, q = lane % LG;
  const int64_t v = ((int64_t)blockIdx.x * kThreads + threadIdx.x) >> 6;
  if (v >= j.counts[0]) return;
  const int32_t c = j.kcount[v];
  const int32_t* picks = j.nbr_pad + v * (int64_t)j.fanout;
  const bool active = q < cpr;
  // global row of local src 0 (the first dst node): invalid picks read it
  const int32_t row0 = src_nodes[0];
  auto row_of = [&](int32_t key) -> int64_t {
    const int32_t r = key >= 0 && (int64_t)key < n_rows ? key : row0;
    return (r >= 0 && (int64_t)r < n_rows ? (int64_t)r : -1);
  };
  float acc[C::VEC];
  zero<C::VEC>(acc);
  int32_t r = g;
  for (; r + G < c; r += 2 * G) {
    const int64_t a0 = row_of(picks[r]), a1 = row_of(picks[r + G]);
    float x0[C::VEC], x1[C::VEC];
    if (active) {
      C::load(H, (a0 < 0 ? 0 : a0) * ld16 + q, x0);
      C::load(H, (a1 < 0 ? 0 : a1) * ld16 + q, x1);
      if (a0 < 0) zero<C::VEC>(x0);
      if (a1 < 0) zero<C::VEC>(x1);
#pragma unroll
      for (int i = 0; i < C::VEC; ++i) acc[i] += 1.f * x0[i] + 1.f * x1[i];
    }
  }
  if (r < c && active) {
    const int64_t a0 = row_of(picks[r]);
    float x0[C::VEC];
    C::load(H, (a0 < 0 ? 0 : a0) * ld16 + q, x0);
    if (a0 < 0) zero<C::VEC>(x0);
#pragma unroll
    for (int i = 0; i < C::VEC; ++i) acc[i] += 1.f * x0[i];
  }
#pragma unroll
  for (int d = LG; d < 64; d <<= 1) {
#pragma unroll
    for (int i = 0; i < C::VEC; ++i) acc[i] += __shfl_xor(acc[i], d, 64);
  }
  if (g != 0 || !active) return;
  float* row = out + v * (int64_t)out_ld;
  const float scale = c > 0 ? 1.f / (float)c : 0.f;
  const int32_t sv = src_nodes[v];
  const bool oks = sv >= 0 && (int64_t)sv < n_rows;
  float xs[C::VEC];
  C::load(H, (oks ? (int64_t)sv : 0) * ld16 + q, xs);
  if (!oks) zero<C::VEC>(xs);
  float4* so = reinterpret_cast<float4*>(row) + q * (C::VEC / 4);
#pragma unroll
  for (int i = 0; i < C::VEC / 4; ++i)
    so[i] = make_float4(xs[4 * i], xs[4 * i + 1], xs[4 * i + 2], xs[4 * i + 3]);
  float4* ao = reinterpret_cast<float4*>(row + cpr * C::VEC) + q * (C::VEC / 4);
#pragma unroll
  for (int i = 0; i < C::VEC / 4; ++i)
    ao[i] = make_float4(acc[4 * i] * scale, acc[4 * i + 1] * scale, acc[4 * i + 2] * scale,
                        acc[4 * i + 3] * scale);
}

// dH[u] += w_e dAgg[v] for every edge (v, u) (+ GCN self edge), fp32 atomics.
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
    rs = rsqrtf((float)(c + 1));
    if (g == 0) {
      const float w = rs * rsqrtf((float)b.occ[v]);
      float* o = dH + v * (int64_t)F;
#pragma unroll
      for (int j = 0; j < NV; ++j) {
        const int f = q + j * LG;
        if (f < F) unsafeAtomicAdd(o + f, w * d[j]);
      }
    }
  }
  for (int32_t e = e0 + g; e < e1; e += G) {
    const int32_t u = b.indices[e];
    const float w = KIND == GNN_GCN ? rs * rsqrtf((float)b.occ[u]) : rs;
    float* o = dH + (int64_t)u * F;
#pragma unroll
    for (int j = 0; j < NV; ++j) {
      const int f = q + j * LG;
      if (f < F) unsafeAtomicAdd(o + f, w * d[j]);
    }
  }
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
                       float* agg, int32_t out_ld, hipStream_t st) {
  const int32_t es = DT == GNN_F32 ? 4 : 2;
  const int32_t cpr = F * es / 16;
  const int lg = pow2_at_least(cpr);
  const unsigned grid = (unsigned)std::max<int64_t>(1, ceil_div((int64_t)blk->cap_dst * 64, kThreads));
  BlockDev b = dev_view(blk);
  auto go = [&](auto kernel) {
    launch("aggregate", kernel, grid, kThreads, 0, st, b, H, cpr, map, agg, out_ld);
  };
  switch (lg) {
    case 1: go(aggregate_kernel<DT, KIND, 1>); break;
    case 2: go(aggregate_kernel<DT, KIND, 2>); break;
    case 4: go(aggregate_kernel<DT, KIND, 4>); break;
    case 8: go(aggregate_kernel<DT, KIND, 8>); break;
    case 16: go(aggregate_kernel<DT, KIND, 16>); break;
    case 32: go(aggregate_kernel<DT, KIND, 32>); break;
    case 64: go(aggregate_kernel<DT, KIND, 64>); break;
    default: return fail(GNN_EINVAL, "aggregate: feature row of %d chunks > 64", cpr);
  }
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
  switch (lg) {
    case 1: go(aggregate_picks_kernel<DT, 1>); break;
    case 2: go(aggregate_picks_kernel<DT, 2>); break;
    case 4: go(aggregate_picks_kernel<DT, 4>); break;
    case 8: go(aggregate_picks_kernel<DT, 8>); break;
    case 16: go(aggregate_picks_kernel<DT, 16>); break;
    case 32: go(aggregate_picks_kernel<DT, 32>); break;
    case 64: go(aggregate_picks_kernel<DT, 64>); break;
    default: return fail(GNN_EINVAL, "aggregate: feature row of %d chunks > 64", cpr);
  }
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
                     int64_t n_rows, int64_t ld_h) {
  if (blk->cap_dst == 0) return GNN_OK;
  const int32_t es = dtype == GNN_F32 ? 4 : 2;
  if (rows && ((ld_h * es) % 16 || ld_h < F)) return fail(GNN_EINVAL, "aggregate: bad row stride");
  const RowMap map{rows, n_rows, rows ? ld_h * es / 16 : 0};
  if (dtype == GNN_F32)
    return kind == GNN_GCN ? dispatch_aggregate<GNN_F32, GNN_GCN>(blk, H, F, map, out, out_ld, st)
                           : dispatch_aggregate<GNN_F32, GNN_SAGE_MEAN>(blk, H, F, map, out, out_ld, st);
  return kind == GNN_GCN ? dispatch_aggregate<GNN_BF16, GNN_GCN>(blk, H, F, map, out, out_ld, st)
                         : dispatch_aggregate<GNN_BF16, GNN_SAGE_MEAN>(blk, H, F, map, out, out_ld, st);
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
  return kind == GNN_GCN ? dispatch_scatter<GNN_GCN>(blk, dAgg, F, dH, st)
                         : dispatch_scatter<GNN_SAGE_MEAN>(blk, dAgg, F, dH, st);
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
