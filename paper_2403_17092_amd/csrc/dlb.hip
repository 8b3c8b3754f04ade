// Dynamic load balancing of mini-batches (paper section 3, Dynamic Load
// Balancer).  Ahead of training, every mini-batch is sampled exactly as the
// training step samples it and its workload is the number of aggregations
// its computation graph needs; batches are then handed to workers by
// estimated workload in proportion to the workers' speeds, and the speeds
// are re-measured after each epoch.
//
// The estimate runs the GPU samplers into a block set of its own and reduces
// each batch's block counts on the device (a one-thread launch per batch), so
// a whole epoch is enqueued without a host round trip.  Assignment and the
// ratio update are host arithmetic.
#include <algorithm>
#include <cmath>
#include <numeric>
#include <vector>

#include "internal.hpp"
#include "relabel.hpp"

namespace gnn {

namespace {

// Workload of one batch: sum over layers of (E + [GCN, GIN, GAT] n_dst) * width, read
// from the counts {n_dst, n_src, E, 0} of the block each layer runs on; the
// edge counts of the listed blocks go to `edges`.
struct WorkJob {
  const int32_t* layer_counts[GNN_MAX_LAYERS];
  int64_t width[GNN_MAX_LAYERS];
  int32_t n_layers;
  int32_t self_rows;  // the aggregation adds each dst row's own features (GCN, GIN)
  const int32_t* edge_counts[GNN_MAX_LAYERS];
  int32_t n_edge_out;
  int64_t* work;   // this batch's entry
  int64_t* edges;  // this batch's row, or null
};

__global__ void __launch_bounds__(64) work_kernel(WorkJob j) {
  if (threadIdx.x != 0) return;
  int64_t w = 0;
  for (int l = 0; l < j.n_layers; ++l) {
    const int32_t* c = j.layer_counts[l];
    w += ((int64_t)c[2] + (j.self_rows ? (int64_t)c[0] : 0)) * j.width[l];
  }
  *j.work = w;
  if (j.edges)
    for (int h = 0; h < j.n_edge_out; ++h) j.edges[h] = j.edge_counts[h][2];
}

int launch_work(const WorkJob& j, hipStream_t st) {
  launch("work", work_kernel, 1, 64, 0, st, j);
  GNN_LAUNCH_CHECK("work estimate");
  return GNN_OK;
}

int check_estimate_model(const gnn_model* m, const char* who) {
  if (!m) return fail(GNN_EINVAL, "%s: null model", who);
  if (m->kind != GNN_SAGE_MEAN && m->kind != GNN_GCN && m->kind != GNN_GIN && m->kind != GNN_GAT)
    return fail(GNN_EINVAL, "%s: bad model kind", who);
  if (m->num_layers < 1 || m->num_layers > GNN_MAX_LAYERS)
    return fail(GNN_EINVAL, "%s: bad layer count", who);
  for (int l = 0; l <= m->num_layers; ++l)
    if (m->dims[l] < 1) return fail(GNN_EINVAL, "%s: dims[%d] < 1", who, l);
  return GNN_OK;
}

int check_csr(const gnn_csr* csr, const char* who) {
  if (!csr || !csr->rowptr || !csr->col) return fail(GNN_EINVAL, "%s: null CSR", who);
  if (csr->rowptr_bits != 32 && csr->rowptr_bits != 64)
    return fail(GNN_EINVAL, "%s: rowptr_bits must be 32 or 64", who);
  if (csr->num_nodes < 0 || csr->num_nodes > INT32_MAX)
    return fail(GNN_EINVAL, "%s: num_nodes out of range", who);
  return check_csr_options(csr, who);
}

// Neighbour sampling: L blocks (hop order), then the sampler's scratch.
struct EstimatePlan {
  gnn_block blocks[GNN_MAX_LAYERS];
  void* sample_ws;
  size_t sample_ws_bytes;
  size_t bytes;
};

int plan_estimate(int32_t B, const int32_t* fanouts, int32_t L, int64_t N, void* ws,
                  EstimatePlan* p) {
  int32_t cd[GNN_MAX_LAYERS], cs[GNN_MAX_LAYERS];
  int64_t ce[GNN_MAX_LAYERS];
  if (int rc = gnn_block_caps(B, fanouts, L, N, cd, cs, ce)) return rc;
  Carver c(ws, SIZE_MAX);
  for (int h = 0; h < L; ++h) {
    gnn_block& b = p->blocks[h];
    b.cap_dst = cd[h];
    b.cap_src = cs[h];
    b.cap_edges = ce[h];
    b.indptr = c.take<int32_t>((size_t)cd[h] + 1);
    b.indices = c.take<int32_t>((size_t)std::max<int64_t>(1, ce[h]));
    b.src_nodes = c.take<int32_t>((size_t)std::max(1, cs[h]));
    b.src_occ = c.take<int32_t>((size_t)std::max(1, cs[h]));
    b.counts = c.take<int32_t>(4);
  }
  p->sample_ws_bytes = sample_scratch_bytes(cd, cs, ce, L, N);
  p->sample_ws = c.take<char>(p->sample_ws_bytes);
  p->bytes = c.off;
  return GNN_OK;
}

// ShaDow: the union block, comp_ptr, the root rows' counts, then the
// extraction's scratch.
struct ShadowEstimatePlan {
  gnn_block sub;
  int32_t* comp_ptr;
  int32_t* readout_counts;
  void* shadow_ws;
  size_t shadow_ws_bytes;
  size_t bytes;
};

int plan_shadow_estimate(int32_t B, int32_t fanout, int32_t hops, void* ws, ShadowEstimatePlan* p) {
  int32_t cn;
  int64_t ce;
  if (int rc = shadow_caps(B, fanout, hops, &cn, &ce)) return rc;
  Carver c(ws, SIZE_MAX);
  gnn_block& b = p->sub;
  b.cap_dst = cn;
  b.cap_src = cn;
  b.cap_edges = ce;
  b.indptr = c.take<int32_t>((size_t)cn + 1);
  b.indices = c.take<int32_t>((size_t)std::max<int64_t>(1, ce));
  b.src_nodes = c.take<int32_t>((size_t)std::max(1, cn));
  b.src_occ = c.take<int32_t>((size_t)std::max(1, cn));
  b.counts = c.take<int32_t>(4);
  p->comp_ptr = c.take<int32_t>((size_t)B + 1);
  p->readout_counts = c.take<int32_t>(4);
  p->shadow_ws_bytes = shadow_scratch_bytes(B, fanout, hops);
  p->shadow_ws = c.take<char>(p->shadow_ws_bytes);
  p->bytes = c.off;
  return GNN_OK;
}

int check_batches(const void* const* ids, const uint64_t* keys, int32_t n, int32_t B,
                  const int64_t* work, const char* who) {
  if (n < 0) return fail(GNN_EINVAL, "%s: n < 0", who);
  if (n > 0 && (!ids || !keys || !work)) return fail(GNN_EINVAL, "%s: null batch arrays", who);
  if (B < 1) return fail(GNN_EINVAL, "%s: empty batch", who);
  for (int32_t i = 0; i < n; ++i)
    if (!ids[i]) return fail(GNN_EINVAL, "%s: batch %d has no node ids", who, i);
  return GNN_OK;
}

}  // namespace

}  // namespace gnn

extern "C" {

size_t gnn_estimate_workspace_bytes(int32_t B, const int32_t* fanouts, int32_t L, int64_t N) {
  gnn::EstimatePlan p;
  if (!fanouts || gnn::plan_estimate(B, fanouts, L, N, nullptr, &p) != GNN_OK) return 0;
  return p.bytes;
}

int gnn_estimate_work(const gnn_model* m, const gnn_csr* csr, const int32_t* const* seeds,
                      const uint64_t* keys, int32_t n, int32_t B, const int32_t* fanouts,
                      int64_t* work, int64_t* edges, void* ws, size_t ws_bytes, void* stream) {
  using namespace gnn;
  const char* who = "gnn_estimate_work";
  if (int rc = check_estimate_model(m, who)) return rc;
  if (int rc = check_csr(csr, who)) return rc;
  if (!fanouts || !ws) return fail(GNN_EINVAL, "%s: null pointer", who);
  if (int rc = check_batches(reinterpret_cast<const void* const*>(seeds), keys, n, B, work, who))
    return rc;
  const int32_t L = m->num_layers;
  EstimatePlan p;
  if (int rc = plan_estimate(B, fanouts, L, csr->num_nodes, ws, &p)) return rc;
  if (p.bytes > ws_bytes) return fail(GNN_EWORKSPACE, "%s: workspace %zu < %zu bytes", who, ws_bytes, p.bytes);
  hipStream_t st = as_stream(stream);
  WorkJob j{};
  j.n_layers = L;
  j.self_rows = m->kind != GNN_SAGE_MEAN;
  j.n_edge_out = L;
  for (int l = 1; l <= L; ++l) {
    j.layer_counts[l - 1] = p.blocks[L - l].counts;  // layer l runs on hop L + 1 - l
    j.width[l - 1] = m->kind == GNN_GAT ? m->dims[l] : m->dims[l - 1];  // GAT sums transformed rows
  }
  for (int h = 0; h < L; ++h) j.edge_counts[h] = p.blocks[h].counts;
  for (int32_t i = 0; i < n; ++i) {
    // consecutive calls on one scratch: all but the first of every
    // kChainCalls skip the sampler's begin launch
    if (int rc = sample_blocks_impl(csr, seeds[i], B, fanouts, L, keys[i], p.blocks, p.sample_ws,
                                    p.sample_ws_bytes, nullptr, 0, nullptr, st, nullptr,
                                    i % (int32_t)kChainCalls != 0))
      return rc;
    j.work = work + i;
    j.edges = edges ? edges + (int64_t)i * L : nullptr;
    if (int rc = launch_work(j, st)) return rc;
  }
  return GNN_OK;
}

size_t gnn_shadow_estimate_workspace_bytes(int32_t B, int32_t fanout, int32_t hops) {
  gnn::ShadowEstimatePlan p;
  if (gnn::plan_shadow_estimate(B, fanout, hops, nullptr, &p) != GNN_OK) return 0;
  return p.bytes;
}

int gnn_shadow_estimate_work(const gnn_model* m, const gnn_csr* csr, const int32_t* const* roots,
                             const uint64_t* keys, int32_t n, int32_t B, int32_t fanout,
                             int32_t hops, int64_t* work, int64_t* edges, void* ws,
                             size_t ws_bytes, void* stream) {
  using namespace gnn;
  const char* who = "gnn_shadow_estimate_work";
  if (int rc = check_estimate_model(m, who)) return rc;
  if (int rc = check_csr(csr, who)) return rc;
  if (!ws) return fail(GNN_EINVAL, "%s: null workspace", who);
  if (int rc = check_batches(reinterpret_cast<const void* const*>(roots), keys, n, B, work, who))
    return rc;
  const int32_t L = m->num_layers;
  ShadowEstimatePlan p;
  if (int rc = plan_shadow_estimate(B, fanout, hops, ws, &p)) return rc;
  if (p.bytes > ws_bytes) return fail(GNN_EWORKSPACE, "%s: workspace %zu < %zu bytes", who, ws_bytes, p.bytes);
  hipStream_t st = as_stream(stream);
  // layers 1..L-1 run on the union block, layer L on the roots' rows
  WorkJob j{};
  j.n_layers = L;
  j.self_rows = m->kind != GNN_SAGE_MEAN;
  for (int l = 1; l <= L; ++l) {
    j.layer_counts[l - 1] = l < L ? p.sub.counts : p.readout_counts;
    j.width[l - 1] = m->kind == GNN_GAT ? m->dims[l] : m->dims[l - 1];  // GAT sums transformed rows
  }
  j.n_edge_out = 2;
  j.edge_counts[0] = p.sub.counts;
  j.edge_counts[1] = p.readout_counts;
  for (int32_t i = 0; i < n; ++i) {
    if (int rc = sample_shadow_impl(csr, roots[i], B, fanout, hops, keys[i], &p.sub, p.comp_ptr,
                                    p.readout_counts, p.shadow_ws, p.shadow_ws_bytes, st))
      return rc;
    j.work = work + i;
    j.edges = edges ? edges + (int64_t)i * 2 : nullptr;
    if (int rc = launch_work(j, st)) return rc;
  }
  return GNN_OK;
}

int gnn_dlb_assign(const int64_t* work, int32_t n, const double* ratio, int32_t k, int32_t* worker,
                   int64_t* load) {
  using namespace gnn;
  if (n < 0 || k < 1 || !ratio || (n > 0 && (!work || !worker)))
    return fail(GNN_EINVAL, "gnn_dlb_assign: bad arguments");
  double rsum = 0.0;
  for (int32_t j = 0; j < k; ++j) {
    if (!(ratio[j] >= 0.0) || !std::isfinite(ratio[j]))
      return fail(GNN_EINVAL, "gnn_dlb_assign: ratio[%d] must be finite and >= 0", j);
    rsum += ratio[j];
  }
  if (!(rsum > 0.0)) return fail(GNN_EINVAL, "gnn_dlb_assign: ratios sum to 0");
  int64_t total = 0;
  for (int32_t i = 0; i < n; ++i) {
    if (work[i] < 0) return fail(GNN_EINVAL, "gnn_dlb_assign: work[%d] < 0", i);
    if (work[i] > INT64_MAX - total) return fail(GNN_EINVAL, "gnn_dlb_assign: total work overflows");
    total += work[i];
  }
  // target share of each worker; each batch, heaviest first (ties: lower
  // index), goes to the worker furthest below its target (ties: lower id)
  std::vector<double> target(k);
  for (int32_t j = 0; j < k; ++j) target[j] = ratio[j] / rsum * (double)total;
  std::vector<int64_t> acc(k, 0);
  std::vector<int32_t> order(n);
  std::iota(order.begin(), order.end(), 0);
  std::sort(order.begin(), order.end(), [&](int32_t a, int32_t b) {
    return work[a] != work[b] ? work[a] > work[b] : a < b;
  });
  for (int32_t i : order) {
    int32_t best = 0;
    for (int32_t j = 1; j < k; ++j)
      if (target[j] - (double)acc[j] > target[best] - (double)acc[best]) best = j;
    worker[i] = best;
    acc[best] += work[i];
  }
  if (load)
    for (int32_t j = 0; j < k; ++j) load[j] = acc[j];
  return GNN_OK;
}

int gnn_dlb_ratio(const int64_t* load, const double* seconds, const double* prev, int32_t k,
                  double tolerance, double* ratio) {
  using namespace gnn;
  if (k < 1 || !load || !seconds || !prev || !ratio || !(tolerance >= 0.0))
    return fail(GNN_EINVAL, "gnn_dlb_ratio: bad arguments");
  double psum = 0.0;
  for (int32_t j = 0; j < k; ++j) {
    if (!(prev[j] >= 0.0) || !std::isfinite(prev[j]) || load[j] < 0 || !(seconds[j] >= 0.0) ||
        !std::isfinite(seconds[j]))
      return fail(GNN_EINVAL, "gnn_dlb_ratio: bad entry %d", j);
    psum += prev[j];
  }
  if (!(psum > 0.0)) return fail(GNN_EINVAL, "gnn_dlb_ratio: previous ratios sum to 0");
  std::vector<double> out(k);
  for (int32_t j = 0; j < k; ++j) out[j] = prev[j] / psum;
  // workers with work and a time are measured; balanced times keep the ratio
  double tmax = 0.0, tmin = INFINITY, share = 0.0, total_speed = 0.0;
  int32_t measured = 0;
  for (int32_t j = 0; j < k; ++j) {
    if (load[j] > 0 && seconds[j] > 0.0) {
      ++measured;
      tmax = std::max(tmax, seconds[j]);
      tmin = std::min(tmin, seconds[j]);
    }
  }
  if (measured > 0 && tmax - tmin > tolerance * tmax) {
    for (int32_t j = 0; j < k; ++j)
      if (load[j] > 0 && seconds[j] > 0.0) {
        share += out[j];
        total_speed += (double)load[j] / seconds[j];
      }
    for (int32_t j = 0; j < k; ++j)
      if (load[j] > 0 && seconds[j] > 0.0) out[j] = share * ((double)load[j] / seconds[j]) / total_speed;
  }
  for (int32_t j = 0; j < k; ++j) ratio[j] = out[j];
  return GNN_OK;
}

}  // extern "C"
