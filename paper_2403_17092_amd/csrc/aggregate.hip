// Aggregation on a sampled block (Ahat H of paper section 2.1, eqs. (1)-(2)):
// a segmented reduction over the block's CSR rows, and its transpose (the
// scatter-add of the backward pass).
//
// Mapping: one group of LG lanes per dst row (LG = 16-byte chunks per row
// rounded up to a power of two), so a wave reduces 64 / LG rows at once: four
// 128-wide bf16 rows, two 100-wide fp32 rows, one 256-wide fp32 row.  The
// input rows can be addressed through the block's src node ids (the first
// layer then reads the feature table itself, with no separate gathered copy).
// A group first loads its row's edge list, one edge per lane, then issues the
// 128-bit loads of U edges' rows (lane q one chunk of each) before adding
// them in edge order; no reduction across lanes is needed.
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
// The layer-1 aggregation over the last hop's picks: at most this many blocks
// take dst rows (about the workgroups resident at once on 256 CUs), and at
// most this many run the hop's compaction ahead of them.
constexpr int64_t kPicksBlocksMax = 2048;
// the aggregation over a compacted block: at most this many blocks take rows
constexpr int64_t kAggBlocksMax = 2048;
constexpr int64_t kPicksTailBlocksMax = 512;

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
  __device__ static inline void widen(const uint4& x, float* v) {
    v[0] = __uint_as_float(x.x);
    v[1] = __uint_as_float(x.y);
    v[2] = __uint_as_float(x.z);
    v[3] = __uint_as_float(x.w);
  }
  __device__ static inline void load(const void* base, int64_t idx16, float* v) {
    widen(reinterpret_cast<const uint4*>(base)[idx16], v);
  }
};

template <>
struct Chunk<GNN_BF16> {
  static constexpr int VEC = 8;
  __device__ static inline void widen(const uint4& x, float* v) {
    const uint32_t w[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      v[2 * i] = __uint_as_float(w[i] << 16);
      v[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
    }
  }
  __device__ static inline void load(const void* base, int64_t idx16, float* v) {
    widen(reinterpret_cast<const uint4*>(base)[idx16], v);
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

// acc += sum over one row's c edges of w_e H[row_e] (lane q's chunk), for one
// group of LG lanes.  The edge list is taken LG edges at a time, one per lane
// (edge(l, &row, &w) fills the H row, -1 for zeros, and the weight of edge
// l); the group then issues the row loads of U edges before adding them in
// edge order.  Shuffles stay inside the group, whose lanes share c.
template <int DT, int LG, int U, typename EdgeFn>
__device__ __forceinline__ void group_sum_rows(int32_t c, EdgeFn edge, const void* H, int64_t ld16,
                                               int q, bool active, float* acc) {
  using Ck = Chunk<DT>;
  for (int32_t base = 0; base < c; base += LG) {
    const int32_t cc = c - base < LG ? c - base : LG;
    int32_t my_row = -1;
    float my_w = 0.f;
    if (q < cc) edge(base + q, &my_row, &my_w);
    for (int32_t k0 = 0; k0 < cc; k0 += U) {
      // rows in flight are held as loaded (16 bytes each) and widened as added
      uint4 x[U];
      float wv[U];
#pragma unroll
      for (int k = 0; k < U; ++k) {
        const int32_t l = k0 + k;
        const int32_t row = __shfl(my_row, l & (LG - 1), LG);
        const float w = __shfl(my_w, l & (LG - 1), LG);
        const bool ok = l < cc && row >= 0 && active;
        wv[k] = ok ? w : 0.f;
        x[k] = ok ? reinterpret_cast<const uint4*>(H)[(int64_t)row * ld16 + q] : make_uint4(0, 0, 0, 0);
      }
#pragma unroll
      for (int k = 0; k < U; ++k) {
        float xv[Ck::VEC];
        Ck::widen(x[k], xv);
#pragma unroll
        for (int i = 0; i < Ck::VEC; ++i) acc[i] += wv[k] * xv[i];
      }
    }
  }
}

// Rows in flight per group: 8 for a 256-wide fp32 row per wave (16 needed 108
// VGPRs, 4 waves per SIMD, and the 4.3K-row layer-2 aggregation of the
// 111M-node workload took 10.4 us against 9.8), 8 for 32 lanes, 4 for
// narrower groups (8 for the 128-wide bf16 rows of its layer 1: 20.7 ->
// 20.1 us for the launch but a slower pipelined step, 4,641 -> 4,573
// mini-batches/s).
template <int LG, bool FEW>
constexpr int rows_in_flight() {
  return LG >= 32 ? 8 : 4;
}

// VEC values of a chunk stored at element `at` of an output row: fp32
// (16-byte stores) or bf16 rounded to nearest even (VEC = 8: one 16-byte store)
template <int VEC, int OT>
__device__ __forceinline__ void store_chunk(void* row, int64_t at, const float* x) {
  if constexpr (OT == GNN_F32) {
    float4* o = reinterpret_cast<float4*>(static_cast<float*>(row) + at);
#pragma unroll
    for (int i = 0; i < VEC / 4; ++i) o[i] = make_float4(x[4 * i], x[4 * i + 1], x[4 * i + 2], x[4 * i + 3]);
  } else {
    static_assert(VEC == 8, "bf16 rows are written from bf16 chunks");
    uint32_t w[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const __bf16 lo = (__bf16)x[2 * i], hi = (__bf16)x[2 * i + 1];
      w[i] = (uint32_t)__builtin_bit_cast(uint16_t, lo) | ((uint32_t)__builtin_bit_cast(uint16_t, hi) << 16);
    }
    *reinterpret_cast<uint4*>(static_cast<uint16_t*>(row) + at) = make_uint4(w[0], w[1], w[2], w[3]);
  }
}

// X[v] = [H[v] | acc / c] (SAGE: the sum divided once by the edge count, so a
// mean of exactly summed rows is correctly rounded; 0 for c = 0) or
// scale (acc + ws H[v]) (GCN, GIN), lane q's chunk, as OT (fp32, or bf16
// rounded to nearest even)
template <int DT, int KIND, int OT>
__device__ __forceinline__ void write_x(void* row, int32_t cpr, int q, const float* xs,
                                        float* acc, float scale, float ws, int32_t c) {
  using Ck = Chunk<DT>;
  int64_t at = (int64_t)q * Ck::VEC;
  if (KIND == GNN_SAGE_MEAN) {
    store_chunk<Ck::VEC, OT>(row, at, xs);
    at += (int64_t)cpr * Ck::VEC;  // the aggregate starts at column F
    const float fc = (float)c;
#pragma unroll
    for (int i = 0; i < Ck::VEC; ++i) acc[i] = c > 0 ? acc[i] / fc : 0.f;
  } else {
#pragma unroll
    for (int i = 0; i < Ck::VEC; ++i) acc[i] = (acc[i] + ws * xs[i]) * scale;
  }
  store_chunk<Ck::VEC, OT>(row, at, acc);
}

template <int OT>
__device__ __forceinline__ void* out_row(void* out, int64_t v, int32_t out_ld) {
  return OT == GNN_F32 ? (void*)(static_cast<float*>(out) + v * (int64_t)out_ld)
                       : (void*)(static_cast<uint16_t*>(out) + v * (int64_t)out_ld);
}

// Blocks [0, fill_blocks) run the launch's fills first; the others take dst
// rows in a grid-stride loop over the live count.
template <int DT, int KIND, int LG, int U, int OT>
__global__ void __launch_bounds__(kThreads)
aggregate_kernel(BlockDev b, const void* __restrict__ H, int32_t cpr, RowMap map,
                 void* __restrict__ out, int32_t out_ld, int32_t fill_blocks, FillPair fills) {
  if ((int32_t)blockIdx.x < fill_blocks) {
    run_fills(fills, blockIdx.x, fill_blocks, kThreads);
    return;
  }
  using C = Chunk<DT>;
  const int q = lane_id() % LG;
  const int64_t n = b.counts[0];
  const int64_t stride = (int64_t)(gridDim.x - fill_blocks) * (kThreads / LG);
  const bool active = q < cpr;
  const int64_t ld16 = map.rows ? map.ld16 : cpr;
  for (int64_t v = ((int64_t)(blockIdx.x - fill_blocks) * kThreads + threadIdx.x) / LG; v < n;
       v += stride) {
    const int32_t e0 = b.indptr[v], e1 = b.indptr[v + 1];
    const int32_t c = e1 - e0;
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
    group_sum_rows<DT, LG, U>(c, edge, H, ld16, q, active, acc);
    if (!active) continue;
    float scale = 1.f, ws = 0.f;
    if (KIND == GNN_GIN) {
      ws = 1.f;
    } else if (KIND == GNN_GCN) {
      ws = rsqrtf((float)b.occ[v]);  // self edge
      scale = rsqrtf((float)(c + 1));
    }
    write_x<DT, KIND, OT>(out_row<OT>(out, v, out_ld), cpr, q, xs, acc, scale, ws, c);
  }
}

// GraphSAGE-mean aggregation of the last sampled hop straight from its
// padded picks (slot (v, r), r < kcount[v], holds the global id of a sampled
// neighbour of dst v), reading rows of the feature table X: the same sums, in
// the same order, as over the compacted block, but without waiting for the
// compaction, which the first tail_blocks blocks run meanwhile (dispatched
// first, so the compaction's dependent lookups overlap the row reads instead
// of trailing them).  The next wt_blocks blocks write the layer's weights as
// the staged W^T of the bf16 forward that follows (run_wt_job), so that its
// CUs copy them instead of converting W.  The other blocks take dst rows in a
// grid-stride loop over the live count (the grid is sized from the resident
// waves, not from the capacity).  A pick with an invalid id (device error raised by the sampler)
// reads as local row 0, as in the compacted block.
template <int DT, int LG, int U, int OT>
__global__ void __launch_bounds__(kThreads)
aggregate_picks_kernel(SampleTail tail, const int32_t* __restrict__ src_nodes,
                       const void* __restrict__ H, int32_t cpr, int64_t n_rows, int64_t ld16,
                       void* __restrict__ out, int32_t out_ld, int32_t tail_blocks, WtJob wj,
                       int32_t wt_blocks) {
  if ((int32_t)blockIdx.x < tail_blocks) {
    finish_sampling(tail, blockIdx.x, tail_blocks, kThreads);
    return;
  }
  const int32_t lead = tail_blocks + wt_blocks;
  if ((int32_t)blockIdx.x < lead) {
    run_wt_job(wj, blockIdx.x - tail_blocks, wt_blocks, kThreads);
    return;
  }
  using C = Chunk<DT>;
  const IndexJob& j = tail.job;
  const int q = lane_id() % LG;
  const int64_t n = j.counts[0];
  const int64_t stride = (int64_t)(gridDim.x - lead) * (kThreads / LG);
  const bool active = q < cpr;
  auto valid = [&](int32_t r) { return r >= 0 && (int64_t)r < n_rows; };
  // global row of local src 0 (the first dst node): invalid picks read it
  const int32_t row0 = src_nodes[0];
  for (int64_t v = ((int64_t)(blockIdx.x - lead) * kThreads + threadIdx.x) / LG; v < n;
       v += stride) {
    const int32_t* picks = j.nbr_pad + v * (int64_t)j.fanout;
    // a fanout within the group: lane q loads pick q beside the count (the
    // edge list is then read in one pass, edge l by lane l)
    const bool pre = j.fanout <= LG;
    const int32_t pk = pre && q < j.fanout ? picks[q] : -1;
    const int32_t c = j.kcount[v];
    const int32_t sv = src_nodes[v];
    float xs[C::VEC];
    if (active && valid(sv)) C::load(H, (int64_t)sv * ld16 + q, xs);
    else zero<C::VEC>(xs);
    float acc[C::VEC];
    zero<C::VEC>(acc);
    auto edge = [&](int32_t l, int32_t* row, float* w) {
      const int32_t key = pre ? pk : picks[l];
      const int32_t r = valid(key) ? key : row0;
      *row = valid(r) ? r : -1;
      *w = 1.f;
    };
    group_sum_rows<DT, LG, U>(c, edge, H, ld16, q, active, acc);
    if (active)
      write_x<DT, GNN_SAGE_MEAN, OT>(out_row<OT>(out, v, out_ld), cpr, q, xs, acc, 1.f, 0.f, c);
  }
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

// The same backward as a gather over the block's transpose: one group of LG
// lanes per src row u < n_src, each lane CPL 16-byte chunks of the row (chunk
// q + k LG), dH[u] = sum over u's edges (v, u) of w_e dAgg[v] (+ GCN / GIN
// self edge for a dst u), written once (no atomics, no zeroing).  SAGE: rows
// u < n_dst already hold the self path (the dX product wrote them) and are
// added to; the other rows are overwritten.  Rows are taken in a grid-stride
// loop over the live count; the loads that do not depend on the edge list
// (the self row, the mask) are issued before it.
// OUT: 0 the row as is; 1 the row times the ReLU mask (mask > 0), in fp32:
// the next layer down's pre-activation gradient, so that its products read
// it without a mask; 2 the same, written instead as bf16 (nearest even) to
// out16 (same layout), ready for a product on bf16 operands.
template <int KIND, int LG, int CPL, int U, int OUT>
__global__ void __launch_bounds__(kThreads)
scatter_t_kernel(BlockDev b, const int32_t* __restrict__ t_ptr, const int32_t* __restrict__ t_dst,
                 const float* __restrict__ dAgg, float* __restrict__ dH, int32_t F,
                 const float* __restrict__ mask, uint16_t* __restrict__ out16) {
  const int q = lane_id() % LG;
  const int64_t n_src = b.counts[1];
  const int32_t n_dst = b.counts[0];
  const int32_t cpr = F / 4;
  const int64_t stride = (int64_t)gridDim.x * (kThreads / LG);
  for (int64_t u = ((int64_t)blockIdx.x * kThreads + threadIdx.x) / LG; u < n_src; u += stride) {
    // chunk k of this lane: q + k LG (live if below cpr)
    float4 self[CPL], m[CPL];
#pragma unroll
    for (int k = 0; k < CPL; ++k) {
      const int ch = q + k * LG;
      const bool ok = ch < cpr;
      self[k] = make_float4(0.f, 0.f, 0.f, 0.f);
      m[k] = make_float4(0.f, 0.f, 0.f, 0.f);
      if (ok && u < n_dst) {
        if (KIND == GNN_SAGE_MEAN) self[k] = reinterpret_cast<const float4*>(dH + u * (int64_t)F)[ch];
        else self[k] = reinterpret_cast<const float4*>(dAgg + u * (int64_t)F)[ch];
      }
      if (OUT != 0 && ok) m[k] = reinterpret_cast<const float4*>(mask + u * (int64_t)F)[ch];
    }
    const int32_t l0 = t_ptr[u], c = t_ptr[u + 1] - l0;
    float ru = 1.f;
    if (KIND == GNN_GCN) ru = rsqrtf((float)b.occ[u]);
    float acc[CPL][4];
#pragma unroll
    for (int k = 0; k < CPL; ++k) acc[k][0] = acc[k][1] = acc[k][2] = acc[k][3] = 0.f;
    // the edge list LG edges at a time, one per lane, then U rows in flight
    for (int32_t base = 0; base < c; base += LG) {
      const int32_t cc = c - base < LG ? c - base : LG;
      int32_t my_v = 0;
      float my_w = 0.f;
      if (q < cc) {
        my_v = t_dst[l0 + base + q];
        const int32_t cv = b.indptr[my_v + 1] - b.indptr[my_v];
        my_w = KIND == GNN_GCN ? ru * rsqrtf((float)(cv + 1)) : (KIND == GNN_GIN ? 1.f : 1.f / (float)cv);
      }
      for (int32_t k0 = 0; k0 < cc; k0 += U) {
        float4 x[U][CPL];
        float wv[U];
#pragma unroll
        for (int e = 0; e < U; ++e) {
          const int32_t l = k0 + e;
          const int32_t v = __shfl(my_v, l & (LG - 1), LG);
          const float w = __shfl(my_w, l & (LG - 1), LG);
          wv[e] = l < cc ? w : 0.f;
#pragma unroll
          for (int k = 0; k < CPL; ++k) {
            const int ch = q + k * LG;
            x[e][k] = l < cc && ch < cpr ? reinterpret_cast<const float4*>(dAgg + (int64_t)v * F)[ch]
                                         : make_float4(0.f, 0.f, 0.f, 0.f);
          }
        }
#pragma unroll
        for (int e = 0; e < U; ++e)
#pragma unroll
          for (int k = 0; k < CPL; ++k) {
            acc[k][0] += wv[e] * x[e][k].x;
            acc[k][1] += wv[e] * x[e][k].y;
            acc[k][2] += wv[e] * x[e][k].z;
            acc[k][3] += wv[e] * x[e][k].w;
          }
      }
    }
    float ws = 1.f;  // weight of the self row (SAGE: the self path as written)
    if (KIND == GNN_GCN && u < n_dst)
      ws = ru * rsqrtf((float)(b.indptr[u + 1] - b.indptr[u] + 1));
#pragma unroll
    for (int k = 0; k < CPL; ++k) {
      const int ch = q + k * LG;
      if (ch >= cpr) continue;
      float y[4] = {acc[k][0], acc[k][1], acc[k][2], acc[k][3]};
      if (u < n_dst) {
        y[0] += ws * self[k].x;
        y[1] += ws * self[k].y;
        y[2] += ws * self[k].z;
        y[3] += ws * self[k].w;
      }
      if constexpr (OUT != 0) {
        y[0] = m[k].x > 0.f ? y[0] : 0.f;
        y[1] = m[k].y > 0.f ? y[1] : 0.f;
        y[2] = m[k].z > 0.f ? y[2] : 0.f;
        y[3] = m[k].w > 0.f ? y[3] : 0.f;
      }
      if constexpr (OUT == 2) {
        uint32_t w2[2];
#pragma unroll
        for (int i = 0; i < 2; ++i) {
          const __bf16 lo = (__bf16)y[2 * i], hi = (__bf16)y[2 * i + 1];
          w2[i] = (uint32_t)__builtin_bit_cast(uint16_t, lo) | ((uint32_t)__builtin_bit_cast(uint16_t, hi) << 16);
        }
        *reinterpret_cast<uint2*>(out16 + u * (int64_t)F + 4 * ch) = make_uint2(w2[0], w2[1]);
      } else {
        *reinterpret_cast<float4*>(dH + u * (int64_t)F + 4 * ch) = make_float4(y[0], y[1], y[2], y[3]);
      }
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

template <int DT, int KIND, int OT>
int dispatch_aggregate(const gnn_block* blk, const void* H, int32_t F, const RowMap& map,
                       void* agg, int32_t out_ld, const FillPair& fills, hipStream_t st) {
  const int32_t es = DT == GNN_F32 ? 4 : 2;
  const int32_t cpr = F * es / 16;
  const int lg = pow2_at_least(cpr);
  const int64_t ablocks = std::min<int64_t>(
      kAggBlocksMax, std::max<int64_t>(1, ceil_div((int64_t)blk->cap_dst * lg, kThreads)));
  const int64_t fblocks = fill_blocks(fills, kThreads);
  const unsigned grid = (unsigned)(ablocks + fblocks);
  BlockDev b = dev_view(blk);
  auto go = [&](auto kernel) {
    launch("aggregate", kernel, grid, kThreads, 0, st, b, H, cpr, map, agg, out_ld,
           (int32_t)fblocks, fills);
  };
  // rows in flight: more while the rows fit the resident waves
  const bool few = blk->cap_dst <= kFewRows;
#define GNN_AGG_CASE(N)                                                          \
  case N:                                                                        \
    if (few) go(aggregate_kernel<DT, KIND, N, rows_in_flight<N, true>(), OT>);   \
    else go(aggregate_kernel<DT, KIND, N, rows_in_flight<N, false>(), OT>);      \
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

template <int DT, int OT>
int dispatch_aggregate_picks(const SampleTail& tail, int32_t cap_dst, const int32_t* src_nodes,
                             const void* H, int32_t F, int64_t n_rows, int64_t ld16, void* out,
                             int32_t out_ld, hipStream_t st, const WtJob* wt) {
  const int32_t es = DT == GNN_F32 ? 4 : 2;
  const int32_t cpr = F * es / 16;
  const int lg = pow2_at_least(cpr);
  const int64_t ablocks = std::min<int64_t>(kPicksBlocksMax,
                                            std::max<int64_t>(1, ceil_div((int64_t)cap_dst * lg, kThreads)));
  const int64_t slots = (int64_t)cap_dst * tail.job.fanout;
  const int64_t tblocks = std::min<int64_t>(kPicksTailBlocksMax, std::max<int64_t>(1, ceil_div(slots, kThreads * 4)));
  const int32_t wblocks = wt ? kWtJobBlocks : 0;
  const WtJob wj = wt ? *wt : WtJob{};
  auto go = [&](auto kernel) {
    launch("aggregate", kernel, (unsigned)(ablocks + tblocks + wblocks), kThreads, 0, st, tail,
           src_nodes, H, cpr, n_rows, ld16, out, out_ld, (int32_t)tblocks, wj, wblocks);
  };
  const bool few = cap_dst <= kFewRows;
#define GNN_AGG_CASE(N)                                                          \
  case N:                                                                        \
    if (few) go(aggregate_picks_kernel<DT, N, rows_in_flight<N, true>(), OT>);   \
    else go(aggregate_picks_kernel<DT, N, rows_in_flight<N, false>(), OT>);      \
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
                     void* out, int32_t out_ld, hipStream_t st, const int32_t* rows,
                     int64_t n_rows, int64_t ld_h, const FillPair& fills, int32_t out_dtype) {
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
  if (out_dtype == GNN_BF16) {
    // bf16 rows of a bf16 input (layer 1 of a bf16-feature GraphSAGE / GCN step)
    if (dtype != GNN_BF16 || kind == GNN_GIN || out_ld % 8)
      return fail(GNN_EINVAL, "aggregate: bf16 output needs bf16 input rows, kind SAGE or GCN");
    if (kind == GNN_GCN)
      return dispatch_aggregate<GNN_BF16, GNN_GCN, GNN_BF16>(blk, H, F, map, out, out_ld, fills, st);
    return dispatch_aggregate<GNN_BF16, GNN_SAGE_MEAN, GNN_BF16>(blk, H, F, map, out, out_ld, fills, st);
  }
  if (dtype == GNN_F32) {
    if (kind == GNN_GCN) return dispatch_aggregate<GNN_F32, GNN_GCN, GNN_F32>(blk, H, F, map, out, out_ld, fills, st);
    if (kind == GNN_GIN) return dispatch_aggregate<GNN_F32, GNN_GIN, GNN_F32>(blk, H, F, map, out, out_ld, fills, st);
    return dispatch_aggregate<GNN_F32, GNN_SAGE_MEAN, GNN_F32>(blk, H, F, map, out, out_ld, fills, st);
  }
  if (kind == GNN_GCN) return dispatch_aggregate<GNN_BF16, GNN_GCN, GNN_F32>(blk, H, F, map, out, out_ld, fills, st);
  if (kind == GNN_GIN) return dispatch_aggregate<GNN_BF16, GNN_GIN, GNN_F32>(blk, H, F, map, out, out_ld, fills, st);
  return dispatch_aggregate<GNN_BF16, GNN_SAGE_MEAN, GNN_F32>(blk, H, F, map, out, out_ld, fills, st);
}

int launch_aggregate_picks(const SampleTail& tail, const gnn_block* blk, const void* H,
                           int32_t dtype, int32_t F, int64_t n_rows, int64_t ld_h, void* out,
                           int32_t out_ld, hipStream_t st, int32_t out_dtype, const WtJob* wt) {
  const int32_t es = dtype == GNN_F32 ? 4 : 2;
  if ((ld_h * es) % 16 || ld_h < F) return fail(GNN_EINVAL, "aggregate: bad row stride");
  if (wt && (!wt->W || !wt->wt || (reinterpret_cast<uintptr_t>(wt->wt) & 15) || wt->K <= 0 ||
             thin_fwd_ks(wt->K) == 0 || wt->N <= 0 || wt->N > kThinFwdCols || wt->ldw < wt->N))
    return fail(GNN_EINVAL, "aggregate: bad staged W^T job");
  if (out_dtype == GNN_BF16) {
    if (dtype != GNN_BF16 || out_ld % 8) return fail(GNN_EINVAL, "aggregate: bf16 output needs bf16 input rows");
    return dispatch_aggregate_picks<GNN_BF16, GNN_BF16>(tail, blk->cap_dst, blk->src_nodes, H, F,
                                                        n_rows, ld_h * es / 16, out, out_ld, st, wt);
  }
  if (dtype == GNN_F32)
    return dispatch_aggregate_picks<GNN_F32, GNN_F32>(tail, blk->cap_dst, blk->src_nodes, H, F, n_rows,
                                                      ld_h * es / 16, out, out_ld, st, wt);
  return dispatch_aggregate_picks<GNN_BF16, GNN_F32>(tail, blk->cap_dst, blk->src_nodes, H, F, n_rows,
                                                     ld_h * es / 16, out, out_ld, st, wt);
}

int launch_scatter(const gnn_block* blk, int32_t kind, const float* dAgg, int32_t F, float* dH,
                   hipStream_t st) {
  if (blk->cap_dst == 0) return GNN_OK;
  if (kind == GNN_GCN) return dispatch_scatter<GNN_GCN>(blk, dAgg, F, dH, st);
  if (kind == GNN_GIN) return dispatch_scatter<GNN_GIN>(blk, dAgg, F, dH, st);
  return dispatch_scatter<GNN_SAGE_MEAN>(blk, dAgg, F, dH, st);
}

int launch_scatter_t(const gnn_block* blk, int32_t kind, const int32_t* t_ptr, const int32_t* t_dst,
                     const float* dAgg, int32_t F, float* dH, hipStream_t st, const float* mask,
                     uint16_t* out16) {
  if (blk->cap_src == 0) return GNN_OK;
  if (F % 4 || F > 256) return fail(GNN_EINVAL, "scatter: feature width %d", F);
  if (out16 && !mask) return fail(GNN_EINVAL, "scatter: bf16 output needs its mask");
  if (mask && kind != GNN_SAGE_MEAN && kind != GNN_GCN)
    return fail(GNN_EINVAL, "scatter: masked output for GraphSAGE and GCN only");
  // lanes per src row and 16-byte chunks per lane: rows of up to 16 chunks
  // one per lane, wider rows 16 lanes of 2 or 4 chunks (four rows per wave),
  // with fewer rows in flight the more chunks a lane holds
  const int32_t cpr = F / 4;
  const int lg = std::min(16, pow2_at_least(cpr));
  const int cpl = cpr <= 16 ? 1 : (cpr <= 32 ? 2 : 4);
  const unsigned grid = (unsigned)std::min<int64_t>(
      kAggBlocksMax, std::max<int64_t>(1, ceil_div((int64_t)blk->cap_src * lg, kThreads)));
  BlockDev b = dev_view(blk);
  auto go = [&](auto kernel) {
    launch("scatter", kernel, grid, kThreads, 0, st, b, t_ptr, t_dst, dAgg, dH, F, mask, out16);
  };
  constexpr int SAGE = GNN_SAGE_MEAN;
#define GNN_ST_CASE(N, C, U)                                                               \
  if (lg == N && cpl == C) {                                                               \
    if (mask) {                                                                            \
      if (kind == GNN_GCN) {                                                               \
        if (out16) go(scatter_t_kernel<GNN_GCN, N, C, U, 2>);                              \
        else go(scatter_t_kernel<GNN_GCN, N, C, U, 1>);                                    \
      } else if (out16) {                                                                  \
        go(scatter_t_kernel<SAGE, N, C, U, 2>);                                            \
      } else {                                                                             \
        go(scatter_t_kernel<SAGE, N, C, U, 1>);                                            \
      }                                                                                    \
    } else if (kind == GNN_GCN) go(scatter_t_kernel<GNN_GCN, N, C, U, 0>);                 \
    else if (kind == GNN_GIN) go(scatter_t_kernel<GNN_GIN, N, C, U, 0>);                   \
    else go(scatter_t_kernel<SAGE, N, C, U, 0>);                                           \
    GNN_LAUNCH_CHECK("scatter");                                                           \
    return GNN_OK;                                                                         \
  }
  GNN_ST_CASE(1, 1, 4)
  GNN_ST_CASE(2, 1, 4)
  GNN_ST_CASE(4, 1, 4)
  GNN_ST_CASE(8, 1, 4)
  GNN_ST_CASE(16, 1, 4)
  GNN_ST_CASE(16, 2, 4)
  GNN_ST_CASE(16, 4, 2)
  return fail(GNN_EINVAL, "scatter: feature width %d", F);
#undef GNN_ST_CASE
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
