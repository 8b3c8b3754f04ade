// Layer forward / backward and the whole training step (paper section 2.2:
// sample a computation graph for the batch, fetch features, propagate,
// average the per-root loss gradients, SGD).  Host-side orchestration only:
// every step is a kernel enqueued on the caller's stream, and no count is
// copied back to the host.
#include <algorithm>
#include <cmath>

#include "internal.hpp"

namespace gnn {

namespace {

inline int32_t esize_of(int32_t dtype) { return dtype == GNN_BF16 ? 2 : 4; }

int record(void* const* events, int idx, hipStream_t st) {
  if (!events || !events[idx]) return GNN_OK;
  GNN_HIP_TRY(hipEventRecord(static_cast<hipEvent_t>(events[idx]), st));
  return GNN_OK;
}

// Row stride of a layer's GEMM input X: [H_dst | agg] (SAGE), agg (GCN), or
// [agg | M | pad] (GIN: M = relu(agg W_a), the MLP's hidden rows, padded to
// whole 16-byte chunks).
// GAT keeps only layer 1's input rows (the gathered features, fp32).
inline int32_t x_width(int32_t kind, int32_t F_in, int32_t F_out) {
  if (kind == GNN_GIN) return F_in + (F_out + 3) / 4 * 4;
  return kind == GNN_SAGE_MEAN ? 2 * F_in : F_in;
}
// Rows of a layer's stacked weights: [W_self; W_neigh], W, [W_a; W_b], or
// [W; a_l; a_r] (GAT).
inline int32_t w_rows(int32_t kind, int32_t F_in, int32_t F_out) {
  if (kind == GNN_GAT) return F_in + 2;
  return kind == GNN_SAGE_MEAN ? 2 * F_in : (kind == GNN_GIN ? F_in + F_out : F_in);
}
inline int32_t pad4(int32_t x) { return (x + 3) / 4 * 4; }

// events (optional): bracket the aggregation with GNN_STAGE_AGG1 and the GEMM
// with GNN_STAGE_GEMM1.
// Input rows of a layer: H_in row u, or, with `rows`, H_in row rows[u] of a
// table of n_rows rows with stride ld.  With `picks` (GraphSAGE, the last
// sampled hop) the aggregation reads the hop's padded picks and finishes the
// sampling call in the same launch.
struct RowSource {
  const int32_t* rows = nullptr;
  int64_t n_rows = 0;
  int64_t ld = 0;
  const SampleTail* picks = nullptr;
  FillPair fills;  // done by the same launch (not with `picks`)
};

// Layer 1's GEMM input X is stored in bf16 (rounded to nearest even), and
// the layer's products take bf16 operands, when the features are bf16 and the
// model is GraphSAGE or GCN.
inline bool x1_bf16(const gnn_model* m, int32_t x_dtype) {
  return x_dtype == GNN_BF16 && (m->kind == GNN_SAGE_MEAN || m->kind == GNN_GCN);
}

// out_dtype: X written in fp32, or in bf16 (x1_bf16)
// wt: (with picks) the same launch writes the staged W^T of the bf16 forward
int aggregate_layer(const gnn_block* blk, int32_t kind, const void* H_in, int32_t in_dtype,
                    int32_t F_in, float* X, int32_t K, const RowSource& src, hipStream_t st,
                    int32_t out_dtype = GNN_F32, const WtJob* wt = nullptr) {
  if (kind == GNN_GAT) {
    // GAT aggregates transformed rows: layer 1's part before the weights is
    // the fetch of its input rows
    FillRange fr[2];
    int n = 0;
    for (int r = 0; r < 2; ++r)
      if (src.fills.n[r] > 0) fr[n++] = FillRange{src.fills.p[r], src.fills.n[r], src.fills.v[r]};
    if (n)
      if (int rc = launch_fill(fr, n, st)) return rc;
    return launch_gat_gather(blk, H_in, in_dtype, src.rows, src.n_rows, src.ld, F_in, X, st);
  }
  if (src.picks)
    return launch_aggregate_picks(*src.picks, blk, H_in, in_dtype, F_in, src.n_rows, src.ld, X, K, st,
                                  out_dtype, wt);
  return launch_aggregate(blk, kind, H_in, in_dtype, F_in, X, K, st, src.rows, src.n_rows, src.ld,
                          src.fills, out_dtype);
}

// aggregated: X already holds the aggregation (it is not run again); then
// gemm_fills are done by the GEMM launch (they must not overlap its output).
// bf16: X is stored in bf16 and the product Z = X W takes bf16 operands
// (GraphSAGE and GCN; see x1_bf16).  wt_stage (thin_fwd_wt_elems(K) bf16):
// where an aggregation over the picks writes the bf16 forward's staged W^T.
int layer_fwd_impl(const gnn_block* blk, int32_t kind, const void* H_in, int32_t in_dtype,
                   int32_t F_in, const float* W, int32_t F_out, int32_t relu, float* X,
                   float* H_out, hipStream_t st, void* const* events = nullptr,
                   bool out_zeroed = false, const RowSource& src = RowSource{},
                   bool aggregated = false, const FillPair& gemm_fills = FillPair{},
                   bool bf16 = false, uint16_t* wt_stage = nullptr) {
  const int32_t K = x_width(kind, F_in, F_out);
  const bool xb = bf16 && (kind == GNN_SAGE_MEAN || kind == GNN_GCN);
  const uint16_t* x16 = reinterpret_cast<const uint16_t*>(X);
  const bool thin = xb && thin_fwd_ok(x16, K, W, F_out, H_out, F_out, K, F_out);
  // the staged W^T comes with the aggregation launch when it reads the picks
  const bool staged = thin && wt_stage && src.picks && !aggregated;
  const WtJob wj{W, F_out, K, F_out, wt_stage};
  if (int rc = record(events, 2 * GNN_STAGE_AGG1, st)) return rc;
  if (!aggregated)
    if (int rc = aggregate_layer(blk, kind, H_in, in_dtype, F_in, X, K, src, st,
                                 xb ? GNN_BF16 : GNN_F32, staged ? &wj : nullptr))
      return rc;
  if (int rc = record(events, 2 * GNN_STAGE_AGG1 + 1, st)) return rc;
  // Z = X W, X = [H_dst | agg] (SAGE) or agg (GCN), W the stacked weights
  MatView A, B;
  OutView C;
  A.p = X;
  A.ld = K;
  A.bf16 = xb;
  A.p16 = reinterpret_cast<const uint16_t*>(X);
  B.p = W;
  B.ld = F_out;
  C.p0 = H_out;
  C.ld0 = F_out;
  C.fills = gemm_fills;
  C.bf16 = xb;
  if (int rc = record(events, 2 * GNN_STAGE_GEMM1, st)) return rc;
  int32_t k_dim = K;
  if (kind == GNN_GIN) {
    // the MLP's first product, M = relu(agg W_a), into X's columns after agg;
    // the second reads M with W_b
    C.p0 = X + F_in;
    C.ld0 = K;
    if (int rc = launch_gemm(A, B, C, blk->cap_dst, F_out, F_in, blk->counts, nullptr, 1, 0,
                             "gemm_fwd", st))
      return rc;
    A.p = X + F_in;
    B.p = W + (int64_t)F_in * F_out;
    C = OutView{};
    C.p0 = H_out;
    C.ld0 = F_out;
    k_dim = F_out;
  }
  // bf16 layer 1 of GraphSAGE / GCN: W^T staged once per CU, X rows streamed
  // (writes every live row, so a zeroed output needs no split)
  if (thin) {
    if (int rc = launch_thin_fwd(x16, K, W, F_out, H_out, F_out, blk->cap_dst, blk->counts, K, F_out,
                                 relu != 0, gemm_fills, "gemm_fwd", st, staged ? wt_stage : nullptr))
      return rc;
    return record(events, 2 * GNN_STAGE_GEMM1 + 1, st);
  }
  // without ReLU into a zeroed output the reduction can be split (short, wide
  // layers such as the output layer then still fill the GPU); chunks of at
  // least 128 keep the atomic partials per output few (1024 x 512 x 172:
  // 13.3 us at 64, 10.9 us at 128)
  const bool split = !relu && out_zeroed;
  if (int rc = launch_gemm(A, B, C, blk->cap_dst, F_out, k_dim, blk->counts, nullptr,
                           split ? 2 : (relu ? 1 : 0), split ? 128 : 0, "gemm_fwd", st))
    return rc;
  return record(events, 2 * GNN_STAGE_GEMM1 + 1, st);
}

// dW must be zero on entry (the reduction over rows is atomic).
// dZ_mask (optional): this layer's ReLU output H_out; dZ is then the
// gradient w.r.t. H_out and is masked by H_out > 0 as the GEMMs read it.
// mask_relu: mask the produced dH_in by H_in > 0 in a pass of its own (the
// training step leaves that to the next layer's GEMMs instead).
// tr (optional): the block's transpose; the input gradient is then gathered
// over it (every row written once) instead of scattered with atomics into
// zeroed rows.
// dM (GIN): [cap_dst x x_width] rows for the gradient of the MLP's hidden
// rows, kept in M's layout (columns F_in ..) so that M masks it in place.
// bf16: X is stored in bf16 and the weight gradient X^T dZ takes bf16
// operands (GraphSAGE and GCN); dZ16: dZ itself as bf16 (already masked), or
// null.  dH16 (with dH16_mask): the gathered input gradient goes there as
// bf16 times (dH16_mask > 0) -- the layer below's pre-activation gradient for
// its bf16 weight-gradient product -- instead of to dH_in.  dH_mask (GraphSAGE
// and GCN, with the transpose): the gathered dH_in is written times
// (dH_mask > 0), the layer below's pre-activation gradient, so that its
// products read it unmasked.
int layer_bwd_impl(const gnn_block* blk, int32_t kind, int32_t F_in, const float* X,
                   const float* H_in, const float* W, int32_t F_out, const float* dZ,
                   const float* dZ_mask, float* dW, float* dH_in, int32_t mask_relu, float* dAgg,
                   hipStream_t st, const BlockTranspose* tr = nullptr, float* dM = nullptr,
                   bool bf16 = false, const uint16_t* dZ16 = nullptr,
                   const float* dH16_mask = nullptr, uint16_t* dH16 = nullptr,
                   const float* dH_mask = nullptr) {
  const int32_t K = x_width(kind, F_in, F_out);
  // rows of the weight block whose gradient the next product forms, and the
  // gradient it contracts with (GIN: of the MLP's first product)
  int32_t kw = w_rows(kind, F_in, F_out);
  const float* g = dZ;
  int64_t g_ld = F_out;
  const float* g_mask = dZ_mask;
  if (kind == GNN_GIN) {
    if (!dM) return fail(GNN_EINVAL, "GIN backward: no staging rows");
    const float* M = X + F_in;
    // dW_b = M^T dZ
    MatView A, B;
    OutView C;
    A.p = M;
    A.ld = K;
    A.trans = 1;
    B.p = dZ;
    B.ld = F_out;
    B.mask = dZ_mask;
    C.p0 = dW + (int64_t)F_in * F_out;
    C.ld0 = F_out;
    if (int rc = launch_gemm(A, B, C, F_out, F_out, blk->cap_dst, nullptr, blk->counts, 2, 256,
                             "gemm_dw", st))
      return rc;
    // dM = dZ W_b^T; the products below read it masked by M > 0 (= dP)
    MatView A2, B2;
    OutView C2;
    A2.p = dZ;
    A2.ld = F_out;
    A2.mask = dZ_mask;
    B2.p = W + (int64_t)F_in * F_out;
    B2.ld = F_out;
    B2.trans = 1;
    C2.p0 = dM + F_in;
    C2.ld0 = K;
    if (int rc = launch_gemm(A2, B2, C2, blk->cap_dst, F_out, F_out, blk->counts, nullptr, 0, 0,
                             "gemm_dx", st))
      return rc;
    kw = F_in;
    g = dM + F_in;
    g_ld = K;
    g_mask = M;
  }
  // dW = X^T dZ (GIN: dW_a = agg^T dP); the reduction runs over the n_dst rows
  const bool xb = bf16 && (kind == GNN_SAGE_MEAN || kind == GNN_GCN);
  MatView A, B;
  OutView C;
  A.p = X;
  A.ld = K;
  A.trans = 1;
  A.bf16 = xb;
  A.p16 = reinterpret_cast<const uint16_t*>(X);
  B.p = g;
  B.ld = g_ld;
  B.mask = g_mask;
  if (xb && dZ16) {
    B.bf16 = 1;
    B.p16 = dZ16;
    B.mask = nullptr;
  }
  C.p0 = dW;
  C.ld0 = F_out;
  C.bf16 = xb;
  if (!dH_in)
    return launch_gemm(A, B, C, kw, F_out, blk->cap_dst, nullptr, blk->counts, 2, 256, "gemm_dw", st);

  // dX = dZ W^T: SAGE -> [dH_in[:n_dst] | dAgg] (self path written in place),
  // GCN -> dAgg, GIN -> dAgg = dP W_a^T.  The same launch zeroes the rows of
  // dH_in the scatter adds into and the product does not write: [n_dst, n_src)
  // for SAGE, all for GCN and GIN.
  MatView A2, B2;
  OutView C2;
  A2.p = g;
  A2.ld = g_ld;
  A2.mask = g_mask;
  B2.p = W;
  B2.ld = F_out;
  B2.trans = 1;
  const bool gather = tr && tr->t_ptr;
  if (!gather) {
    C2.zero_p = dH_in;
    C2.zero_ld = F_in;
    C2.zero_cols = F_in;
    C2.zero_hi = blk->counts + 1;
    C2.zero_cap = blk->cap_src;
  }
  if (kind == GNN_SAGE_MEAN) {
    C2.p0 = dH_in;
    C2.ld0 = F_in;
    C2.p1 = dAgg;
    C2.ld1 = F_in;
    C2.axis = 1;
    C2.split = F_in;
    C2.zero_lo = blk->counts;
  } else {
    C2.p0 = dAgg;
    C2.ld0 = F_in;
  }
  // dW and dX are independent: one launch of both grids (GIN's come in its
  // own order above).  dW's rows in chunks of at least 1024 (fewer atomic
  // partials, more of the GPU left to dX: 4335-row layer of the 111M-node
  // workload, 41.0 -> 35.5 us against chunks of 256)
  const GemmSpec dw{A, B, C, kw, F_out, blk->cap_dst, nullptr, blk->counts, 2, 1024, "gemm_dw"};
  const GemmSpec dx{A2, B2, C2, blk->cap_dst, kw, F_out, blk->counts, nullptr, 0, 0, "gemm_dx"};
  if (kind == GNN_GIN) {
    if (int rc = launch_gemm(A, B, C, kw, F_out, blk->cap_dst, nullptr, blk->counts, 2, 256,
                             "gemm_dw", st))
      return rc;
    if (int rc = launch_gemm(A2, B2, C2, blk->cap_dst, kw, F_out, blk->counts, nullptr, 0, 0,
                             "gemm_dx", st))
      return rc;
  } else if (int rc = launch_gemm_pair(dw, dx, "gemm_bwd", st)) {
    return rc;
  }
  if (dH16 && !gather) return fail(GNN_EINVAL, "layer backward: bf16 input gradient needs the transpose");
  if (int rc = gather ? launch_scatter_t(blk, kind, tr->t_ptr, tr->t_dst, dAgg, F_in, dH_in, st,
                                         dH16 ? dH16_mask : dH_mask, dH16)
                      : launch_scatter(blk, kind, dAgg, F_in, dH_in, st))
    return rc;
  if (mask_relu) return launch_relu_mask(blk, H_in, F_in, dH_in, st);
  return GNN_OK;
}

int check_block(const gnn_block* b, const char* who) {
  if (!b || !b->indptr || !b->indices || !b->src_nodes || !b->src_occ || !b->counts)
    return fail(GNN_EINVAL, "%s: null block array", who);
  if (b->cap_dst < 0 || b->cap_src < b->cap_dst || b->cap_edges < 0)
    return fail(GNN_EINVAL, "%s: bad block capacities", who);
  return GNN_OK;
}

int check_width(int32_t F, int32_t dtype, const char* who) {
  if (F <= 0 || F > 256) return fail(GNN_EINVAL, "%s: width %d not in [1, 256]", who, F);
  if (dtype == GNN_F32 ? (F % 4) : (F % 8)) return fail(GNN_EINVAL, "%s: width %d not a 16-byte multiple", who, F);
  return GNN_OK;
}

int check_model(const gnn_model* m, const char* who) {
  if (!m || !m->weights) return fail(GNN_EINVAL, "%s: null model", who);
  if (m->kind != GNN_SAGE_MEAN && m->kind != GNN_GCN && m->kind != GNN_GIN && m->kind != GNN_GAT)
    return fail(GNN_EINVAL, "%s: bad model kind", who);
  if (m->num_layers < 1 || m->num_layers > GNN_MAX_LAYERS) return fail(GNN_EINVAL, "%s: bad layer count", who);
  for (int l = 0; l <= m->num_layers; ++l)
    if (m->dims[l] < 1 || m->dims[l] > 256) return fail(GNN_EINVAL, "%s: dims[%d] not in [1, 256]", who, l);
  for (int l = 1; l < m->num_layers; ++l)
    if (m->dims[l] % 4) return fail(GNN_EINVAL, "%s: hidden width dims[%d] must be a multiple of 4", who, l);
  if (const gnn_optimizer* o = m->opt) {
    if (o->kind != GNN_OPT_SGD && o->kind != GNN_OPT_ADAM) return fail(GNN_EINVAL, "%s: bad optimizer", who);
    if (o->kind == GNN_OPT_ADAM &&
        (!o->m || !o->v || !(o->beta1 >= 0.0 && o->beta1 < 1.0) || !(o->beta2 >= 0.0 && o->beta2 < 1.0) ||
         !(o->eps > 0.0) || o->steps < 0))
      return fail(GNN_EINVAL, "%s: bad Adam state", who);
  }
  return GNN_OK;
}

// Workspace plan of one training step.  `layer_blk[l-1]` is the block layer
// l runs on: for neighbour sampling the block of hop L + 1 - l; for ShaDow the
// square union block, and for the last layer its prefix of root rows.
struct StepPlan {
  int32_t L;
  bool shadow;
  int32_t cap_dst[GNN_MAX_LAYERS], cap_src[GNN_MAX_LAYERS];
  int64_t cap_edges[GNN_MAX_LAYERS];
  gnn_block blocks[GNN_MAX_LAYERS];  // NS: hop order; ShaDow: [0] union, [1] root rows
  // NS: transposes of the blocks of hops h < L - 1 (the layers >= 2 gather
  // their input gradients over them); ShaDow: none (atomic scatter)
  BlockTranspose tr[GNN_MAX_LAYERS];
  const gnn_block* layer_blk[GNN_MAX_LAYERS];
  int32_t layer_rows[GNN_MAX_LAYERS];  // row capacity of layer l's output
  int32_t* comp_ptr;
  void* sample_ws;
  size_t sample_ws_bytes;
  float* x[GNN_MAX_LAYERS];
  float* h[GNN_MAX_LAYERS];
  float* dweights;
  float* dlogits;
  float* dh[2];
  float* dagg;
  float* dm;  // GIN: the hidden rows' gradient (see layer_bwd_impl)
  // x1_bf16: layer 1's pre-activation gradient as bf16, masked (written by
  // layer 2's transpose gather), or null
  uint16_t* dz16;
  int32_t x1_dtype;  // storage of layer 1's GEMM input x[0] (GNN_F32 or GNN_BF16)
  // with dz16: layer 1's weight gradient as dw1_nparts partial sums over
  // chunks of its rows (summed by the optimizer launch)
  float* dw1_part;
  int32_t dw1_nparts;
  // x1_bf16 GraphSAGE: the staged W^T of layer 1's bf16 forward, written by
  // the aggregation launch that reads the last hop's picks
  uint16_t* w1t;
  // GAT: per layer the transformed rows T [cap_src x pad4(F_out)], the scores
  // [cap_src x 2] and the softmax statistics [cap_dst x 2]; the gradients dT
  // and (ds_l, ds_r) of the layer being differentiated
  float* z[GNN_MAX_LAYERS];
  float* s[GNN_MAX_LAYERS];
  float* stats[GNN_MAX_LAYERS];
  float* dz;
  float* ds;
  float* hh;    // GAT layer 1: [H^T ds_l | H^T ds_r] (F_in x 2)
  float* part;  // GAT: per-workgroup column sums (gat_colsum_part_floats())
  float* row_loss;
  // output layer and loss in one launch (head.hip); its weight gradient comes
  // as per-tile partials
  bool head;
  float* head_part;
  float* head_xch;
  int32_t* head_sync;
  size_t bytes;
};

void carve_block(Carver& c, gnn_block& b) {
  b.indptr = c.take<int32_t>((size_t)b.cap_dst + 1);
  b.indices = c.take<int32_t>((size_t)std::max<int64_t>(1, b.cap_edges));
  b.src_nodes = c.take<int32_t>((size_t)std::max(1, b.cap_src));
  b.src_occ = c.take<int32_t>((size_t)std::max(1, b.cap_src));
  b.counts = c.take<int32_t>(4);
}

// Activations and gradients of the model part (shared by both samplers).
const float* weight_ptr(const gnn_model* m, int layer);

void carve_model(Carver& c, const gnn_model* m, int32_t x_dtype, int32_t B, StepPlan* p) {
  const int L = p->L;
  size_t dh_elems = 1, dagg_elems = 1, dm_elems = 0, dz_elems = 0, ds_elems = 0;
  const bool gat = m->kind == GNN_GAT;
  for (int l = 1; l <= L; ++l) {
    const gnn_block* b = p->layer_blk[l - 1];
    const int32_t rows = std::max(1, b->cap_dst);
    const int32_t xw = x_width(m->kind, m->dims[l - 1], m->dims[l]);
    p->layer_rows[l - 1] = rows;
    p->z[l - 1] = p->s[l - 1] = p->stats[l - 1] = nullptr;
    if (gat) {
      const size_t src_rows = (size_t)std::max(1, b->cap_src);
      p->z[l - 1] = c.take<float>(src_rows * pad4(m->dims[l]));
      p->s[l - 1] = c.take<float>(src_rows * 2);
      p->stats[l - 1] = c.take<float>((size_t)rows * 2);
      dz_elems = std::max(dz_elems, src_rows * pad4(m->dims[l]));
      // (layer 1 keeps its attention-weighted input rows there instead)
      if (l == 1) dz_elems = std::max(dz_elems, (size_t)rows * m->dims[0]);
      ds_elems = std::max(ds_elems, src_rows * 2);
      if (l > 1) p->x[l - 1] = nullptr;
    }
    // layer 1's input belongs to the block slot (set by the plan)
    if (l > 1 && !gat) p->x[l - 1] = c.take<float>((size_t)rows * xw);
    if (m->kind == GNN_GIN) dm_elems = std::max(dm_elems, (size_t)rows * xw);
    p->h[l - 1] = c.take<float>((size_t)rows * m->dims[l]);
    if (l >= 2) {
      dh_elems = std::max(dh_elems, (size_t)b->cap_src * m->dims[l - 1]);
      dagg_elems = std::max(dagg_elems, (size_t)b->cap_dst * m->dims[l - 1]);
    }
  }
  p->dweights = c.take<float>((size_t)gnn_num_params(m));
  p->dlogits = c.take<float>((size_t)std::max(1, B) * m->dims[L]);
  p->dh[0] = c.take<float>(dh_elems);
  p->dh[1] = c.take<float>(dh_elems);
  p->dagg = c.take<float>(dagg_elems);
  p->dm = dm_elems ? c.take<float>(dm_elems) : nullptr;
  p->x1_dtype = x1_bf16(m, x_dtype) ? GNN_BF16 : GNN_F32;
  // (sized by the condition, not the pointer: a size query carves from null)
  const bool dz16 = x1_bf16(m, x_dtype) && L >= 2;
  p->dz16 = dz16 ? c.take<uint16_t>((size_t)std::max(1, p->layer_blk[0]->cap_dst) * m->dims[1])
                 : nullptr;
  p->dw1_nparts = dz16 ? thin_dw_parts(p->layer_blk[0]->cap_dst) : 0;
  p->dw1_part = dz16 ? c.take<float>((size_t)p->dw1_nparts *
                                     w_rows(m->kind, m->dims[0], m->dims[1]) * m->dims[1])
                     : nullptr;
  const int32_t k1 = x_width(m->kind, m->dims[0], m->dims[1]);
  const bool w1t = x1_bf16(m, x_dtype) && m->kind == GNN_SAGE_MEAN && thin_fwd_ks(k1) > 0 &&
                   m->dims[1] <= kThinFwdCols;
  p->w1t = w1t ? c.take<uint16_t>((size_t)thin_fwd_wt_elems(k1)) : nullptr;
  p->dz = dz_elems ? c.take<float>(dz_elems) : nullptr;
  p->ds = ds_elems ? c.take<float>(ds_elems) : nullptr;
  p->hh = gat ? c.take<float>(2 * (size_t)m->dims[0]) : nullptr;
  p->part = gat ? c.take<float>(gat_colsum_part_floats()) : nullptr;
  p->row_loss = c.take<float>((size_t)std::max(1, B));
  // (the partials are part of the workspace whenever the widths allow the
  // fused output layer; it is used if the layer's weights are also aligned.
  // A GIN output layer is two products: it runs unfused)
  const bool head_dims = L >= 2 && (m->kind == GNN_SAGE_MEAN || m->kind == GNN_GCN) &&
                         m->dims[L] >= kHeadMinClasses &&
                         m->dims[L] <= kHeadMaxClasses;
  p->head_part = head_dims ? c.take<float>((size_t)head_part_elems(B, x_width(m->kind, m->dims[L - 1], m->dims[L]),
                                                                   m->dims[L]))
                           : nullptr;
  p->head_xch = head_dims ? c.take<float>((size_t)head_xch_elems(B)) : nullptr;
  p->head_sync = head_dims ? c.take<int32_t>((size_t)head_sync_words(B)) : nullptr;
  p->head = head_dims && (reinterpret_cast<uintptr_t>(weight_ptr(m, L)) & 15) == 0;
}

// The workspace holds two slots of blocks (a batch can be sampled into one
// while the model trains on the other), then the sampler's scratch and the
// model's buffers; `slot` selects the blocks the plan points at.
constexpr int kSlots = 2;

int plan_step(const gnn_model* m, int32_t x_dtype, int32_t B, const int32_t* fanouts, int64_t N,
              void* ws, size_t ws_bytes, StepPlan* p, int32_t slot = 0) {
  const int L = m->num_layers;
  p->L = L;
  p->shadow = false;
  p->comp_ptr = nullptr;
  if (slot < 0 || slot >= kSlots) return fail(GNN_EINVAL, "training step: slot %d not 0 or 1", slot);
  if (int rc = gnn_block_caps(B, fanouts, L, N, p->cap_dst, p->cap_src, p->cap_edges)) return rc;
  Carver c(ws, ws_bytes);
  for (int s = 0; s < kSlots; ++s) {
    for (int h = 0; h < L; ++h) {
      gnn_block b;
      b.cap_dst = p->cap_dst[h];
      b.cap_src = p->cap_src[h];
      b.cap_edges = p->cap_edges[h];
      carve_block(c, b);
      BlockTranspose t;
      if (h < L - 1) {
        t.t_ptr = c.take<int32_t>((size_t)b.cap_src + 1);
        t.t_cur = c.take<int32_t>((size_t)std::max(1, b.cap_src));
        t.t_dst = c.take<int32_t>((size_t)std::max<int64_t>(1, b.cap_edges));
      }
      if (s == slot) {
        p->blocks[h] = b;
        p->tr[h] = t;
      }
    }
    // layer 1's input (the aggregation of the outermost hop) belongs to the slot
    // (GAT: the gathered input rows of every src node)
    const int32_t x1_rows = m->kind == GNN_GAT ? p->cap_src[L - 1] : p->cap_dst[L - 1];
    float* x1 = c.take<float>((size_t)std::max(1, x1_rows) * x_width(m->kind, m->dims[0], m->dims[1]));
    if (s == slot) p->x[0] = x1;
  }
  for (int l = 1; l <= L; ++l) p->layer_blk[l - 1] = &p->blocks[L - l];
  p->sample_ws_bytes = sample_scratch_bytes(p->cap_dst, p->cap_src, p->cap_edges, L, N);
  p->sample_ws = c.take<char>(p->sample_ws_bytes);
  carve_model(c, m, x_dtype, B, p);
  p->bytes = c.off;
  return GNN_OK;
}

int plan_shadow_step(const gnn_model* m, int32_t x_dtype, int32_t B, int32_t fanout, int32_t hops,
                     void* ws, size_t ws_bytes, StepPlan* p, int32_t slot = 0) {
  const int L = m->num_layers;
  p->L = L;
  p->shadow = true;
  if (slot < 0 || slot >= kSlots) return fail(GNN_EINVAL, "training step: slot %d not 0 or 1", slot);
  int32_t cn;
  int64_t ce;
  if (int rc = shadow_caps(B, fanout, hops, &cn, &ce)) return rc;
  Carver c(ws, ws_bytes);
  for (int s = 0; s < kSlots; ++s) {
    gnn_block sub;
    sub.cap_dst = cn;
    sub.cap_src = cn;
    sub.cap_edges = ce;
    carve_block(c, sub);
    // the root rows are the prefix of the union block; only the counts differ
    gnn_block ro = sub;
    ro.cap_dst = B;
    ro.counts = c.take<int32_t>(4);
    int32_t* comp = c.take<int32_t>((size_t)B + 1);
    // layer 1's input (ShaDow: L >= 2, so layer 1 runs on the union block)
    // (GAT: the gathered input rows of every src node of the union)
    const int32_t x1_rows = L >= 2 || m->kind == GNN_GAT ? cn : B;
    float* x1 = c.take<float>((size_t)std::max(1, x1_rows) * x_width(m->kind, m->dims[0], m->dims[1]));
    if (s == slot) {
      p->blocks[0] = sub;
      p->blocks[1] = ro;
      p->comp_ptr = comp;
      p->x[0] = x1;
    }
  }
  for (int l = 1; l <= L; ++l) p->layer_blk[l - 1] = l < L ? &p->blocks[0] : &p->blocks[1];
  p->sample_ws_bytes = shadow_scratch_bytes(B, fanout, hops);
  p->sample_ws = c.take<char>(p->sample_ws_bytes);
  carve_model(c, m, x_dtype, B, p);
  p->bytes = c.off;
  return GNN_OK;
}

// Zero fills a step needs before its first gradient accumulation: the
// weight gradient (split-K atomics) and, with the fused output layer, its
// exchange counters, else the logits (split-K output layer).
int step_fills(const gnn_model* m, const StepPlan& p, FillRange* fr) {
  const int L = p.L;
  fr[0] = FillRange{p.dweights, gnn_num_params(m), 0};
  if (p.head) fr[1] = FillRange{p.head_sync, (int64_t)head_sync_words(p.layer_rows[L - 1]), 0};
  else fr[1] = FillRange{p.h[L - 1], (int64_t)p.layer_rows[L - 1] * m->dims[L], 0};
  return 2;
}

const float* weight_ptr(const gnn_model* m, int layer) {
  const float* w = m->weights;
  for (int l = 1; l < layer; ++l) w += (int64_t)w_rows(m->kind, m->dims[l - 1], m->dims[l]) * m->dims[l];
  return w;
}

int mark_event(void* const* events, int stage, int end, hipStream_t st) {
  return record(events, 2 * stage + end, st);
}

// The update of every training step: the loss mean and SGD or Adam on the
// step's weight gradient (plus the fused output layer's partials, if any).
int update_weights(const gnn_model* m, const StepPlan& p, float lr, int32_t B, float* loss_out,
                   void* const* events, hipStream_t st, const GradParts& parts) {
  if (int rc = mark_event(events, GNN_STAGE_BACKWARD, 1, st)) return rc;
  if (int rc = mark_event(events, GNN_STAGE_SGD, 0, st)) return rc;
  AdamJob adam;
  gnn_optimizer* opt = m->opt;
  if (opt && opt->kind == GNN_OPT_ADAM) {
    const double t = (double)(opt->steps + 1);
    adam = AdamJob{opt->m,
                   opt->v,
                   (float)opt->beta1,
                   (float)(1.0 - opt->beta1),
                   (float)opt->beta2,
                   (float)(1.0 - opt->beta2),
                   (float)opt->eps,
                   (float)(1.0 / (1.0 - std::pow(opt->beta1, t))),
                   (float)(1.0 / (1.0 - std::pow(opt->beta2, t)))};
  }
  if (int rc = launch_sgd(m->weights, p.dweights, gnn_num_params(m), lr, p.row_loss, B, loss_out, st,
                          parts, adam))
    return rc;
  if (adam.m) ++opt->steps;
  return mark_event(events, GNN_STAGE_SGD, 1, st);
}

// GAT layer 1 has no input gradient, so its weight gradient dW = H^T dT is
// formed without dT: dT_u = sum_v alpha_vu dOut_v + ds_r[u] a_r + [u < n_dst]
// ds_l[u] a_l gives dW = G^T dOut + (H^T ds_l) a_l^T + (H^T ds_r) a_r^T, with
// G_v = sum_u alpha_vu H_u the attention-weighted input rows (an aggregation
// over the block, no atomics).  The score gradients come from the same
// backward pass over the edges with its dT output switched off.
// zeroed: ds and hh were zeroed by an earlier launch of the step.
int gat_layer1_bwd(const gnn_model* m, const StepPlan& p, const gnn_block* blk, const float* dout,
                   int64_t ld_do, const float* mask, hipStream_t st, bool zeroed) {
  const int32_t Fi = m->dims[0], Fo = m->dims[1], ldt = pad4(Fo);
  const float* W = weight_ptr(m, 1);
  const float* a = W + (int64_t)Fi * Fo;
  float* dw = p.dweights + (W - m->weights);
  const float* hin = p.x[0];
  float* G = p.dz;
  if (!zeroed) {
    const FillRange zr[2] = {{p.ds, (int64_t)std::max(1, blk->cap_src) * 2, 0}, {p.hh, (int64_t)Fi * 2, 0}};
    if (int rc = launch_fill(zr, 2, st)) return rc;
  }
  if (int rc = launch_gat_attend_bwd(blk, p.z[0], ldt, p.s[0], p.stats[0], dout, ld_do, mask, Fo,
                                     nullptr, p.ds, st))
    return rc;
  // G: the forward's attention (same scores, so the same weights) over H
  if (int rc = launch_gat_attend(blk, hin, Fi, p.s[0], Fi, 0, G, p.stats[0], st)) return rc;
  // [da_l; da_r] = [ds_l | ds_r]^T T and hh = H^T [ds_l | ds_r]
  if (int rc = launch_gat_colsum2(blk->counts + 1, blk->cap_src, p.ds, p.z[0], ldt, Fo, p.part,
                                  dw + (int64_t)Fi * Fo, Fo, 1, st))
    return rc;
  if (int rc = launch_gat_colsum2(blk->counts + 1, blk->cap_src, p.ds, hin, Fi, Fi, p.part, p.hh, 1, 2, st))
    return rc;
  // dW = G^T dOut (dOut masked by the layer's ReLU output), reduced over the dst rows
  MatView A, Bm;
  OutView C;
  A.p = G;
  A.ld = Fi;
  A.trans = 1;
  Bm.p = dout;
  Bm.ld = ld_do;
  Bm.mask = mask;
  C.p0 = dw;
  C.ld0 = Fo;
  if (int rc = launch_gemm(A, Bm, C, Fi, Fo, blk->cap_dst, nullptr, blk->counts, 2, 256, "gemm_dw", st))
    return rc;
  // dW += hh [a_l; a_r]
  MatView A2, B2;
  OutView C2;
  A2.p = p.hh;
  A2.ld = 2;
  B2.p = a;
  B2.ld = Fo;
  C2.p0 = dw;
  C2.ld0 = Fo;
  return launch_gemm(A2, B2, C2, Fi, Fo, 2, nullptr, nullptr, 2, 0, "gemm_dw", st);
}

// GAT forward and backward (gat.hip for the attention; GEMMs for T = H W and
// the weight and input gradients).  Layer 1's input rows are the features of
// its src nodes, widened to fp32 into x[0] (beside the sampling when
// x1_ready).  Input gradients flow as dH_in = dT W^T over the block's src
// rows; the next layer down masks them by its ReLU output as it reads them.
int run_gat(const gnn_model* m, const StepPlan& p, const void* X, int32_t x_dtype, int64_t ld_x,
            int64_t num_nodes, const int32_t* labels, const int32_t* label_rows, int32_t B,
            void* const* events, hipStream_t st, const FillPair& fills, bool x1_ready, bool x_local) {
  const int L = p.L;
  const int32_t* dims = m->dims;
  if (int rc = mark_event(events, GNN_STAGE_GATHER, 0, st)) return rc;
  if (!x1_ready) {
    RowSource src{x_local ? nullptr : p.layer_blk[0]->src_nodes, num_nodes, ld_x};
    src.fills = fills;
    if (int rc = aggregate_layer(p.layer_blk[0], GNN_GAT, X, x_dtype, dims[0], p.x[0], dims[0], src, st))
      return rc;
  } else {
    FillRange fr[2];
    int n = 0;
    for (int r = 0; r < 2; ++r)
      if (fills.n[r] > 0) fr[n++] = FillRange{fills.p[r], fills.n[r], fills.v[r]};
    if (n)
      if (int rc = launch_fill(fr, n, st)) return rc;
  }
  if (int rc = mark_event(events, GNN_STAGE_GATHER, 1, st)) return rc;
  for (int l = 1; l <= L; ++l) {
    const gnn_block* blk = p.layer_blk[l - 1];
    const int32_t Fi = dims[l - 1], Fo = dims[l], ldt = pad4(Fo);
    const float* W = weight_ptr(m, l);
    const float* hin = l == 1 ? p.x[0] : p.h[l - 2];
    if (l == 1)
      if (int rc = mark_event(events, GNN_STAGE_GEMM1, 0, st)) return rc;
    MatView A, Bm;
    OutView C;
    A.p = hin;
    A.ld = Fi;
    Bm.p = W;
    Bm.ld = Fo;
    C.p0 = p.z[l - 1];
    C.ld0 = ldt;
    if (l == L && L >= 2) {
      // the output layer's backward buffers are zeroed by this launch
      const FillRange zr[2] = {{p.dz, (int64_t)std::max(1, blk->cap_src) * ldt, 0},
                               {p.ds, (int64_t)std::max(1, blk->cap_src) * 2, 0}};
      C.fills = fill_pair(zr, 2);
    }
    if (int rc = launch_gemm(A, Bm, C, blk->cap_src, Fo, Fi, blk->counts + 1, nullptr, 0, 0, "gemm_fwd", st))
      return rc;
    if (l == 1) {
      if (int rc = mark_event(events, GNN_STAGE_GEMM1, 1, st)) return rc;
      if (int rc = mark_event(events, GNN_STAGE_AGG1, 0, st)) return rc;
    }
    if (int rc = launch_gat_scores(blk, p.z[l - 1], ldt, W + (int64_t)Fi * Fo, Fo, p.s[l - 1], st))
      return rc;
    if (int rc = launch_gat_attend(blk, p.z[l - 1], ldt, p.s[l - 1], Fo, l < L, p.h[l - 1],
                                   p.stats[l - 1], st))
      return rc;
    if (l == 1) {
      if (int rc = mark_event(events, GNN_STAGE_AGG1, 1, st)) return rc;
      if (int rc = mark_event(events, GNN_STAGE_FWD_REST, 0, st)) return rc;
    }
  }
  if (int rc = launch_softmax_xent(p.h[L - 1], labels, num_nodes, label_rows, B, dims[L], dims[L],
                                   p.dlogits, p.row_loss, st))
    return rc;
  if (int rc = mark_event(events, GNN_STAGE_FWD_REST, 1, st)) return rc;
  if (int rc = mark_event(events, GNN_STAGE_BACKWARD, 0, st)) return rc;
  const float* dout = p.dlogits;
  int64_t ld_do = dims[L];
  const float* mask = nullptr;
  for (int l = L; l >= 1; --l) {
    const gnn_block* blk = p.layer_blk[l - 1];
    const int32_t Fi = dims[l - 1], Fo = dims[l], ldt = pad4(Fo);
    const float* W = weight_ptr(m, l);
    const float* hin = l == 1 ? p.x[0] : p.h[l - 2];
    float* dw = p.dweights + (W - m->weights);
    const int32_t src_rows = std::max(1, blk->cap_src);
    if (l == 1) {
      if (int rc = gat_layer1_bwd(m, p, blk, dout, ld_do, mask, st, L >= 2)) return rc;
      break;
    }
    if (l < L) {  // (layer L's were zeroed by its forward product)
      const FillRange zr[2] = {{p.dz, (int64_t)src_rows * ldt, 0}, {p.ds, (int64_t)src_rows * 2, 0}};
      if (int rc = launch_fill(zr, 2, st)) return rc;
    }
    if (int rc = launch_gat_attend_bwd(blk, p.z[l - 1], ldt, p.s[l - 1], p.stats[l - 1], dout, ld_do,
                                       mask, Fo, p.dz, p.ds, st))
      return rc;
    if (int rc = launch_gat_score_grad(blk, W + (int64_t)Fi * Fo, Fo, p.ds, p.dz, ldt, st)) return rc;
    // [da_l; da_r] = [ds_l | ds_r]^T T (ds_l is 0 past the dst rows)
    if (int rc = launch_gat_colsum2(blk->counts + 1, blk->cap_src, p.ds, p.z[l - 1], ldt, Fo, p.part,
                                    dw + (int64_t)Fi * Fo, Fo, 1, st))
      return rc;
    // dW = H_in^T dT
    MatView A, Bm;
    OutView C;
    A.p = hin;
    A.ld = Fi;
    A.trans = 1;
    Bm.p = p.dz;
    Bm.ld = ldt;
    C.ld0 = Fo;
    C.p0 = dw;
    if (int rc = launch_gemm(A, Bm, C, Fi, Fo, blk->cap_src, nullptr, blk->counts + 1, 2, 256,
                             "gemm_dw", st))
      return rc;
    // dH_in = dT W^T over the src rows: the next layer down's output gradient
    MatView A2, B2;
    OutView C2;
    A2.p = p.dz;
    A2.ld = ldt;
    B2.p = W;
    B2.ld = Fo;
    B2.trans = 1;
    C2.p0 = p.dh[l & 1];
    C2.ld0 = Fi;
    if (l == 2) {
      // layer 1's ds and hh (ds is read no more by this layer; dT is, and is not zeroed)
      const gnn_block* b1 = p.layer_blk[0];
      const FillRange zr[2] = {{p.ds, (int64_t)std::max(1, b1->cap_src) * 2, 0},
                               {p.hh, (int64_t)dims[0] * 2, 0}};
      C2.fills = fill_pair(zr, 2);
    }
    if (int rc = launch_gemm(A2, B2, C2, blk->cap_src, Fi, Fo, blk->counts + 1, nullptr, 0, 0, "gemm_dx", st))
      return rc;
    dout = p.dh[l & 1];
    ld_do = Fi;
    mask = p.h[l - 2];
  }
  return GNN_OK;
}

// Forward, loss on rows 0..B-1 of the last layer (labels[label_rows[i]]),
// backward, SGD, on blocks the step's sampler has filled.  The first layer
// reads its input rows straight from the feature table X through the src
// node ids of its block (the features of the sampled nodes are never copied
// out first).
// `fills` (if no `tail`): zero fills the step needs, done by the first launch.
// x1_ready: layer 1's input X already holds its aggregation (done beside the
// sampling); the model pass then starts with layer 1's GEMM.
// x_local: X holds the feature rows of layer 1's src nodes by local id (a
// fetched copy, row stride dims[0]) instead of the whole table.
int run_model(const gnn_model* m, const StepPlan& p, const void* X, int32_t x_dtype, int64_t ld_x,
              int64_t num_nodes, const int32_t* labels, const int32_t* label_rows, int32_t B,
              float lr, float* loss_out, void* const* events, const SampleTail* tail,
              hipStream_t st, const FillPair& fills = FillPair{}, bool x1_ready = false,
              bool x_local = false) {
  if (m->kind == GNN_GAT) {
    if (int rc = run_gat(m, p, X, x_dtype, ld_x, num_nodes, labels, label_rows, B, events, st, fills,
                         x1_ready, x_local))
      return rc;
    return update_weights(m, p, lr, B, loss_out, events, st, GradParts{});
  }
  const int L = p.L;
  const int32_t* dims = m->dims;
  // the feature fetch is part of the layer-1 aggregation: an empty stage
  if (int rc = mark_event(events, GNN_STAGE_GATHER, 0, st)) return rc;
  if (int rc = mark_event(events, GNN_STAGE_GATHER, 1, st)) return rc;
  for (int l = 1; l <= L; ++l) {
    const void* hin = l == 1 ? X : p.h[l - 2];
    const int32_t dt = l == 1 ? x_dtype : GNN_F32;
    // layer 1: rows of X through the block's src node ids (or the sampled
    // hop's picks, if the sampling call's last step was left to this launch)
    RowSource src{l == 1 && !x_local ? p.layer_blk[0]->src_nodes : nullptr, num_nodes, ld_x,
                  l == 1 ? tail : nullptr};
    const bool aggregated = l == 1 && x1_ready;
    FillPair gemm_fills;
    if (l == 1 && !x1_ready) src.fills = fills;
    if (aggregated) {
      // the first launch is this GEMM: it takes the fills, unless its own
      // output is one of them (one layer: the split-K logits)
      if (L >= 2) gemm_fills = fills;
      else {
        FillRange fr[2];
        int n = 0;
        for (int r = 0; r < 2; ++r)
          if (fills.n[r] > 0) fr[n++] = FillRange{fills.p[r], fills.n[r], fills.v[r]};
        if (int rc = launch_fill(fr, n, st)) return rc;
      }
    }
    if (l == 2) {
      if (int rc = mark_event(events, GNN_STAGE_FWD_REST, 0, st)) return rc;
    }
    if (l == L && p.head) {
      // aggregation only; the product is the head's
      if (int rc = aggregate_layer(p.layer_blk[l - 1], m->kind, hin, dt, dims[l - 1], p.x[l - 1],
                                   x_width(m->kind, dims[l - 1], dims[l]), src, st))
        return rc;
      continue;
    }
    if (int rc = layer_fwd_impl(p.layer_blk[l - 1], m->kind, hin, dt, dims[l - 1], weight_ptr(m, l),
                                dims[l], l < L, p.x[l - 1], p.h[l - 1], st,
                                l == 1 ? events : nullptr, l == L, src, aggregated, gemm_fills,
                                l == 1 && x_dtype == GNN_BF16, l == 1 ? p.w1t : nullptr))
      return rc;
  }
  if (L == 1) {
    if (int rc = mark_event(events, GNN_STAGE_FWD_REST, 0, st)) return rc;
  }
  int top = L;  // layers top .. 1 still to differentiate
  GradParts parts;
  bool dz16_ready = false;  // p.dz16 holds layer 1's pre-activation gradient
  bool dz_masked = false;   // the next layer's dZ already carries its ReLU mask
  if (p.head) {
    // logits, loss, dlogits, the output layer's dW partials and its dX (SAGE:
    // [dH_in rows < n_dst | dAgg]; GCN: dAgg); the rows of dH_in the scatter
    // adds into and the product does not write are zeroed by the same launch
    const gnn_block* blk = p.layer_blk[L - 1];
    const int32_t F = dims[L - 1], K = x_width(m->kind, F, dims[L]);
    float* dh = p.dh[L & 1];
    HeadJob j;
    j.X = p.x[L - 1];
    j.K = K;
    j.W = weight_ptr(m, L);
    j.C = dims[L];
    j.labels = labels;
    j.n_labels = num_nodes;
    j.label_rows = label_rows;
    j.B = B;
    j.logits = p.h[L - 1];
    j.dlogits = p.dlogits;
    j.row_loss = p.row_loss;
    j.dw_part = p.head_part;
    j.xch = p.head_xch;
    j.sync = p.head_sync;
    // neighbour sampling: the input gradient is gathered over the block
    // transpose (every row written once, no zeroing); a ShaDow readout
    // scatters into rows this launch zeroes (its transpose gather, a search
    // for each row's component root, measured slower)
    const BlockTranspose* tr = p.shadow ? nullptr : &p.tr[0];
    const bool gather = tr && tr->t_ptr;
    if (!gather) {
      j.zero_p = dh;
      j.zero_ld = F;
      j.zero_cols = F;
      j.zero_hi = blk->counts + 1;
      j.zero_cap = blk->cap_src;
    }
    if (m->kind == GNN_SAGE_MEAN) {
      j.dx0 = dh;
      j.ld0 = F;
      j.dx1 = p.dagg;
      j.ld1 = F;
      j.split = F;
      j.zero_lo = blk->counts;
    } else {
      j.dx0 = p.dagg;
      j.ld0 = F;
    }
    if (int rc = launch_head(j, st)) return rc;
    if (int rc = mark_event(events, GNN_STAGE_FWD_REST, 1, st)) return rc;
    if (int rc = mark_event(events, GNN_STAGE_BACKWARD, 0, st)) return rc;
    // two layers with a bf16 layer 1: the gather writes layer 1's masked
    // pre-activation gradient in bf16 for its weight-gradient product; else
    // it writes layer L - 1's masked pre-activation gradient in fp32
    const bool to16 = gather && L == 2 && p.dz16;
    if (int rc = gather ? launch_scatter_t(blk, m->kind, tr->t_ptr, tr->t_dst, p.dagg, F, dh, st,
                                           p.h[L - 2], to16 ? p.dz16 : nullptr)
                        : launch_scatter(blk, m->kind, p.dagg, F, dh, st))
      return rc;
    dz16_ready = to16;
    dz_masked = gather && !to16;
    parts.r[0] = GradRange{p.head_part, weight_ptr(m, L) - m->weights, (int64_t)K * dims[L],
                           (int32_t)ceil_div(B, kHeadRows)};
    top = L - 1;
  } else {
    if (int rc = launch_softmax_xent(p.h[L - 1], labels, num_nodes, label_rows, B, dims[L], dims[L],
                                     p.dlogits, p.row_loss, st))
      return rc;
    if (int rc = mark_event(events, GNN_STAGE_FWD_REST, 1, st)) return rc;
    if (int rc = mark_event(events, GNN_STAGE_BACKWARD, 0, st)) return rc;
  }
  // dZ of layer l < L is the gradient w.r.t. its ReLU output, masked by
  // H_l > 0: by the gather of layer l + 1 as it wrote it (dz_masked), else
  // as layer l's GEMMs read it
  const float* dZ = top == L ? p.dlogits : p.dh[L & 1];
  for (int l = top; l >= 1; --l) {
    const float* w = weight_ptr(m, l);
    float* dw = p.dweights + (w - m->weights);
    float* dh = l > 1 ? p.dh[l & 1] : nullptr;
    const float* mask = l < L && !dz_masked ? p.h[l - 1] : nullptr;
    // neighbour sampling: the block's transpose; ShaDow: the union block of a
    // symmetric graph is its own transpose (the readout block, layer L, is
    // not: it keeps the scatter when the output layer runs on its own)
    const gnn_block* lb = p.layer_blk[l - 1];
    const BlockTranspose self_t{lb->indptr, nullptr, lb->indices};
    const BlockTranspose* tr = !p.shadow ? &p.tr[L - l] : (l < L ? &self_t : nullptr);
    // layer 2 over a transpose, with a bf16 layer 1: its gather writes layer
    // 1's masked pre-activation gradient in bf16
    const bool to16 = l == 2 && p.dz16 && tr && tr->t_ptr;
    // otherwise a gather (GraphSAGE, GCN) masks the layer below's gradient
    const bool mask_out = l > 1 && !to16 && tr && tr->t_ptr &&
                          (m->kind == GNN_SAGE_MEAN || m->kind == GNN_GCN);
    if (l == 1 && dz16_ready && p.dw1_part) {
      // bf16 layer 1: dW = X^T dZ as partial sums over chunks of the rows
      const int32_t K = x_width(m->kind, dims[0], dims[1]), kw = w_rows(m->kind, dims[0], dims[1]);
      const uint16_t* x16 = reinterpret_cast<const uint16_t*>(p.x[0]);
      if (thin_dw_ok(x16, K, p.dz16, dims[1], kw, dims[1])) {
        if (int rc = launch_thin_dw(x16, K, p.dz16, dims[1], lb->cap_dst, lb->counts, kw, dims[1],
                                    p.dw1_part, p.dw1_nparts, "gemm_dw", st))
          return rc;
        parts.r[1] = GradRange{p.dw1_part, w - m->weights, (int64_t)kw * dims[1], p.dw1_nparts};
        continue;
      }
    }
    if (int rc = layer_bwd_impl(lb, m->kind, dims[l - 1], p.x[l - 1], nullptr, w, dims[l], dZ, mask,
                                dw, dh, 0, p.dagg, st, l > 1 ? tr : nullptr, p.dm,
                                l == 1 && x_dtype == GNN_BF16, l == 1 && dz16_ready ? p.dz16 : nullptr,
                                to16 ? p.h[0] : nullptr, to16 ? p.dz16 : nullptr,
                                mask_out ? p.h[l - 2] : nullptr))
      return rc;
    if (to16) dz16_ready = true;
    dz_masked = mask_out;
    dZ = dh;
  }
  return update_weights(m, p, lr, B, loss_out, events, st, parts);
}

int check_step_args(const gnn_model* m, const gnn_csr* csr, const void* X, int32_t x_dtype,
                    int64_t ld_x, const int32_t* labels, const int32_t* seeds, int32_t B,
                    float* loss_out, void* ws, const char* who) {
  if (int rc = check_model(m, who)) return rc;
  if (!csr || !X || !labels || !seeds || !loss_out || !ws) return fail(GNN_EINVAL, "%s: null pointer", who);
  if (B < 1) return fail(GNN_EINVAL, "%s: empty batch", who);
  if (x_dtype != GNN_F32 && x_dtype != GNN_BF16) return fail(GNN_EINVAL, "%s: bad dtype", who);
  if (int rc = check_width(m->dims[0], x_dtype, who)) return rc;
  if (!csr->rowptr || !csr->col || (csr->rowptr_bits != 32 && csr->rowptr_bits != 64) ||
      csr->num_nodes < 1 || csr->num_nodes > INT32_MAX)
    return fail(GNN_EINVAL, "%s: bad CSR", who);
  if (ld_x < m->dims[0] || (ld_x * (x_dtype == GNN_BF16 ? 2 : 4)) % 16 ||
      (reinterpret_cast<uintptr_t>(X) & 15))
    return fail(GNN_EINVAL, "%s: feature rows must be 16-byte aligned", who);
  return GNN_OK;
}

void fill_views(const gnn_model* m, const StepPlan& p, gnn_train_views* out) {
  *out = gnn_train_views{};
  const int nb = p.shadow ? 2 : p.L;
  for (int h = 0; h < nb; ++h) out->blocks[h] = p.blocks[h];
  out->xg = nullptr;
  for (int l = 0; l < p.L; ++l) {
    out->x[l] = p.x[l];
    out->x_ld[l] = x_width(m->kind, m->dims[l], m->dims[l + 1]);
    out->x_dtype[l] = l == 0 ? p.x1_dtype : GNN_F32;
    out->h[l] = p.h[l];
  }
  out->dweights = p.dweights;
  out->dlogits = p.dlogits;
  out->comp_ptr = p.comp_ptr;
}

}  // namespace

}  // namespace gnn

namespace gnn {
namespace {

// n steps with the sampling part of step i + 1 on `ss` while step i's model
// part runs on `ms`; ev[0..1]: slot s sampled, ev[2..3]: slot s trained.
template <typename Sample, typename Model>
int run_pipelined(int32_t n, void* const* events, hipStream_t ms, hipStream_t ss, Sample sample,
                  Model model) {
  using namespace gnn;
  if (n <= 0) return GNN_OK;
  if (!events) return fail(GNN_EINVAL, "pipelined steps: null events");
  for (int k = 0; k < 4; ++k)
    if (!events[k]) return fail(GNN_EINVAL, "pipelined steps: null event %d", k);
  auto ev = [&](int k) { return static_cast<hipEvent_t>(events[k]); };
  // the sample stream starts after whatever the model stream holds
  GNN_HIP_TRY(hipEventRecord(ev(2), ms));
  GNN_HIP_TRY(hipStreamWaitEvent(ss, ev(2), 0));
  if (int rc = sample(0, 0, ss)) return rc;
  GNN_HIP_TRY(hipEventRecord(ev(0), ss));
  for (int32_t i = 0; i < n; ++i) {
    const int slot = i & 1;
    if (i + 1 < n) {
      const int nxt = slot ^ 1;
      if (i >= 1) GNN_HIP_TRY(hipStreamWaitEvent(ss, ev(2 + nxt), 0));  // step i - 1 used it
      if (int rc = sample(i + 1, nxt, ss)) return rc;
      GNN_HIP_TRY(hipEventRecord(ev(nxt), ss));
    }
    GNN_HIP_TRY(hipStreamWaitEvent(ms, ev(slot), 0));
    if (int rc = model(i, slot, ms)) return rc;
    GNN_HIP_TRY(hipEventRecord(ev(2 + slot), ms));
  }
  // the model stream ends after the sample stream's last work
  GNN_HIP_TRY(hipEventRecord(ev((n - 1) & 1), ss));
  GNN_HIP_TRY(hipStreamWaitEvent(ms, ev((n - 1) & 1), 0));
  return GNN_OK;
}

}  // namespace
}  // namespace gnn

extern "C" {

int64_t gnn_num_params(const gnn_model* m) {
  if (!m || m->num_layers < 1 || m->num_layers > GNN_MAX_LAYERS) return 0;
  int64_t n = 0;
  for (int l = 1; l <= m->num_layers; ++l)
    n += (int64_t)gnn::w_rows(m->kind, m->dims[l - 1], m->dims[l]) * m->dims[l];
  return n;
}

int gnn_layer_fwd(const gnn_block* blk, int32_t kind, const void* H_in, int32_t in_dtype,
                  int32_t F_in, const float* W, int32_t F_out, int32_t relu, float* X_out,
                  float* H_out, void* stream) {
  using namespace gnn;
  if (int rc = check_block(blk, "gnn_layer_fwd")) return rc;
  if (kind != GNN_SAGE_MEAN && kind != GNN_GCN && kind != GNN_GIN)
    return fail(GNN_EINVAL, "gnn_layer_fwd: bad kind (GAT layers run inside the training steps)");
  if (in_dtype != GNN_F32 && in_dtype != GNN_BF16) return fail(GNN_EINVAL, "gnn_layer_fwd: bad dtype");
  if (int rc = check_width(F_in, in_dtype, "gnn_layer_fwd")) return rc;
  if (F_out < 1 || F_out > 256) return fail(GNN_EINVAL, "gnn_layer_fwd: F_out not in [1, 256]");
  if (!H_in || !W || !X_out || !H_out) return fail(GNN_EINVAL, "gnn_layer_fwd: null pointer");
  hipStream_t st = as_stream(stream);
  if (!relu) {
    FillRange fr[1] = {{H_out, (int64_t)blk->cap_dst * F_out, 0}};
    if (int rc = launch_fill(fr, 1, st)) return rc;
  }
  return layer_fwd_impl(blk, kind, H_in, in_dtype, F_in, W, F_out, relu, X_out, H_out, st, nullptr,
                        !relu);
}

size_t gnn_layer_bwd_workspace_bytes(int32_t cap_dst, int32_t F_in) {
  return (size_t)std::max(1, cap_dst) * std::max(1, F_in) * sizeof(float) + 256;
}

int gnn_layer_bwd(const gnn_block* blk, int32_t kind, int32_t F_in, const float* X,
                  const float* H_in, const float* W, int32_t F_out, const float* dZ, float* dW,
                  float* dH_in, int32_t mask_relu, void* ws, size_t ws_bytes, void* stream) {
  using namespace gnn;
  if (int rc = check_block(blk, "gnn_layer_bwd")) return rc;
  if (kind != GNN_SAGE_MEAN && kind != GNN_GCN && kind != GNN_GIN)
    return fail(GNN_EINVAL, "gnn_layer_bwd: bad kind (GAT layers run inside the training steps)");
  if (int rc = check_width(F_in, GNN_F32, "gnn_layer_bwd")) return rc;
  if (F_out < 1 || F_out > 256) return fail(GNN_EINVAL, "gnn_layer_bwd: F_out not in [1, 256]");
  if (!X || !W || !dZ || !dW) return fail(GNN_EINVAL, "gnn_layer_bwd: null pointer");
  if (dH_in && mask_relu && !H_in) return fail(GNN_EINVAL, "gnn_layer_bwd: the ReLU mask needs H_in");
  const bool gin = kind == GNN_GIN;
  // GIN: dAgg rows, then the hidden rows' gradient in X's layout
  const int32_t ws_cols = gin ? F_in + x_width(kind, F_in, F_out) : F_in;
  if ((dH_in || gin) && (!ws || ws_bytes < gnn_layer_bwd_workspace_bytes(blk->cap_dst, ws_cols)))
    return fail(GNN_EWORKSPACE, "gnn_layer_bwd: workspace too small");
  hipStream_t st = as_stream(stream);
  FillRange fr[1] = {{dW, (int64_t)w_rows(kind, F_in, F_out) * F_out, 0}};
  if (int rc = launch_fill(fr, 1, st)) return rc;
  float* dagg = static_cast<float*>(ws);
  float* dm = gin ? dagg + (size_t)std::max(1, blk->cap_dst) * F_in : nullptr;
  return layer_bwd_impl(blk, kind, F_in, X, H_in, W, F_out, dZ, nullptr, dW, dH_in, mask_relu,
                        dagg, st, nullptr, dm);
}

size_t gnn_train_workspace_bytes(const gnn_model* m, int32_t x_dtype, int32_t B,
                                 const int32_t* fanouts, int64_t N) {
  using namespace gnn;
  if (check_model(m, "gnn_train_workspace_bytes") || !fanouts) return 0;
  StepPlan p;
  if (plan_step(m, x_dtype, B, fanouts, N, nullptr, 0, &p)) return 0;
  return p.bytes;
}

int gnn_train_step_views(const gnn_model* m, int32_t x_dtype, int32_t B, const int32_t* fanouts,
                         int64_t N, void* ws, size_t ws_bytes, gnn_train_views* out) {
  return gnn_train_slot_views(m, x_dtype, B, fanouts, N, ws, ws_bytes, 0, out);
}

int gnn_train_slot_views(const gnn_model* m, int32_t x_dtype, int32_t B, const int32_t* fanouts,
                         int64_t N, void* ws, size_t ws_bytes, int32_t slot, gnn_train_views* out) {
  using namespace gnn;
  if (int rc = check_model(m, "gnn_train_slot_views")) return rc;
  if (!fanouts || !ws || !out) return fail(GNN_EINVAL, "gnn_train_slot_views: null pointer");
  StepPlan p;
  if (int rc = plan_step(m, x_dtype, B, fanouts, N, ws, ws_bytes, &p, slot)) return rc;
  if (p.bytes > ws_bytes) return fail(GNN_EWORKSPACE, "gnn_train_slot_views: workspace too small");
  fill_views(m, p, out);
  return GNN_OK;
}

int gnn_train_step(const gnn_model* m, const gnn_csr* csr, const void* X, int32_t x_dtype,
                   int64_t ld_x, const int32_t* labels, const int32_t* seeds, int32_t B,
                   const int32_t* fanouts, uint64_t rng_key, float lr, float* loss_out, void* ws,
                   size_t ws_bytes, void* stream) {
  return gnn_train_step_ex(m, csr, X, x_dtype, ld_x, labels, seeds, B, fanouts, rng_key, lr,
                           loss_out, ws, ws_bytes, nullptr, stream);
}

int gnn_train_step_ex(const gnn_model* m, const gnn_csr* csr, const void* X, int32_t x_dtype,
                      int64_t ld_x, const int32_t* labels, const int32_t* seeds, int32_t B,
                      const int32_t* fanouts, uint64_t rng_key, float lr, float* loss_out, void* ws,
                      size_t ws_bytes, void* const* events, void* stream) {
  using namespace gnn;
  if (int rc = check_step_args(m, csr, X, x_dtype, ld_x, labels, seeds, B, loss_out, ws,
                               "gnn_train_step"))
    return rc;
  if (!fanouts) return fail(GNN_EINVAL, "gnn_train_step: null fanouts");
  StepPlan p;
  if (int rc = plan_step(m, x_dtype, B, fanouts, csr->num_nodes, ws, ws_bytes, &p)) return rc;
  if (p.bytes > ws_bytes)
    return fail(GNN_EWORKSPACE, "gnn_train_step: workspace %zu < %zu bytes", ws_bytes, p.bytes);
  hipStream_t st = as_stream(stream);
  const int L = p.L;
  // the sampler's first launch also zeroes the weight gradient (atomic
  // split-K) and, without the fused output layer, the logits (split-K
  // output layer)
  FillRange fr[2];
  const int n_fills = step_fills(m, p, fr);
  if (int rc = mark_event(events, GNN_STAGE_SAMPLE, 0, st)) return rc;
  // GraphSAGE: the last hop's edge compaction runs inside the layer-1
  // aggregation launch, which reads the hop's picks directly (GCN weights
  // need the compaction's source degrees first)
  SampleTail tail;
  const bool fuse_tail = m->kind == GNN_SAGE_MEAN;
  if (int rc = sample_blocks_impl(csr, seeds, B, fanouts, L, rng_key, p.blocks, p.sample_ws,
                                  p.sample_ws_bytes, fr, n_fills,
                                  fuse_tail ? &tail : nullptr, st, p.tr))
    return rc;
  if (int rc = mark_event(events, GNN_STAGE_SAMPLE, 1, st)) return rc;
  // the seeds are the dst rows of hop 1, i.e. rows 0..B-1 of the last layer
  return run_model(m, p, X, x_dtype, ld_x, csr->num_nodes, labels, seeds, B, lr, loss_out, events,
                   fuse_tail ? &tail : nullptr, st);
}

}  // extern "C"

namespace gnn {
namespace {
// The cached step's workspace: the step's plan, then the fetched rows of
// layer 1's src nodes and the feature cache's per-call scratch.
struct CachedPlan {
  void* xg;
  void* call_ws;
  size_t call_bytes;
  size_t bytes;
};

int plan_cached(const gnn_model* m, int32_t x_dtype, const StepPlan& p, int32_t num_sets, void* ws,
                CachedPlan* e) {
  const int32_t cap = p.cap_src[p.L - 1];
  const size_t es = x_dtype == GNN_F32 ? 4 : 2;
  Carver c(ws, SIZE_MAX);
  c.off = p.bytes;
  e->xg = c.take<char>((size_t)std::max(1, cap) * m->dims[0] * es);
  e->call_bytes = gnn_gather_cached_workspace_bytes(num_sets, cap);
  if (!e->call_bytes) return fail(GNN_EINVAL, "cached step: bad cache size");
  e->call_ws = c.take<char>(e->call_bytes);
  e->bytes = c.off;
  return GNN_OK;
}
}  // namespace
}  // namespace gnn

extern "C" {

size_t gnn_train_cached_workspace_bytes(const gnn_model* m, int32_t x_dtype, int32_t B,
                                        const int32_t* fanouts, int64_t N, int32_t num_sets) {
  using namespace gnn;
  if (check_model(m, "gnn_train_cached_workspace_bytes") || !fanouts) return 0;
  StepPlan p;
  if (plan_step(m, x_dtype, B, fanouts, N, nullptr, 0, &p)) return 0;
  CachedPlan e;
  if (plan_cached(m, x_dtype, p, num_sets, nullptr, &e)) return 0;
  return e.bytes;
}

int gnn_train_step_cached(const gnn_model* m, const gnn_csr* csr, const void* X, int32_t x_dtype,
                          int64_t ld_x, const gnn_feature_cache* cache, uint64_t* cache_stats,
                          const int32_t* labels, const int32_t* seeds, int32_t B,
                          const int32_t* fanouts, uint64_t rng_key, float lr, float* loss_out,
                          void* ws, size_t ws_bytes, void* stream) {
  using namespace gnn;
  const char* who = "gnn_train_step_cached";
  if (int rc = check_step_args(m, csr, X, x_dtype, ld_x, labels, seeds, B, loss_out, ws, who))
    return rc;
  if (!fanouts || !cache || !cache_stats) return fail(GNN_EINVAL, "%s: null pointer", who);
  if (cache->dtype != x_dtype || cache->width != m->dims[0])
    return fail(GNN_EINVAL, "%s: the cache's rows must match the features' dtype and width", who);
  StepPlan p;
  if (int rc = plan_step(m, x_dtype, B, fanouts, csr->num_nodes, ws, ws_bytes, &p)) return rc;
  CachedPlan e;
  if (int rc = plan_cached(m, x_dtype, p, cache->num_sets, ws, &e)) return rc;
  if (e.bytes > ws_bytes) return fail(GNN_EWORKSPACE, "%s: workspace %zu < %zu bytes", who, ws_bytes, e.bytes);
  hipStream_t st = as_stream(stream);
  const int L = p.L;
  // sampling (its first launch zeroes the gradient buffers), then the rows
  // of the last hop's src nodes through the cache, then the model on them
  FillRange fr[2];
  const int n_fills = step_fills(m, p, fr);
  if (int rc = sample_blocks_impl(csr, seeds, B, fanouts, L, rng_key, p.blocks, p.sample_ws,
                                  p.sample_ws_bytes, fr, n_fills, nullptr, st, p.tr))
    return rc;
  const gnn_block& last = p.blocks[L - 1];
  if (int rc = gnn_gather_cached(cache, X, csr->num_nodes, ld_x, last.src_nodes, last.counts + 1,
                                 last.cap_src, e.xg, m->dims[0], cache_stats, e.call_ws,
                                 e.call_bytes, stream))
    return rc;
  return run_model(m, p, e.xg, x_dtype, m->dims[0], csr->num_nodes, labels, seeds, B, lr, loss_out,
                   nullptr, nullptr, st, FillPair{}, false, true);
}

int gnn_train_sample(const gnn_model* m, const gnn_csr* csr, const void* X, int32_t x_dtype,
                     int64_t ld_x, const int32_t* seeds, int32_t B, const int32_t* fanouts,
                     uint64_t rng_key, void* ws, size_t ws_bytes, int32_t slot, void* stream) {
  using namespace gnn;
  if (int rc = check_model(m, "gnn_train_sample")) return rc;
  if (!csr || !X || !seeds || !fanouts || !ws) return fail(GNN_EINVAL, "gnn_train_sample: null pointer");
  if (B < 1) return fail(GNN_EINVAL, "gnn_train_sample: empty batch");
  if (x_dtype != GNN_F32 && x_dtype != GNN_BF16) return fail(GNN_EINVAL, "gnn_train_sample: bad dtype");
  if (int rc = check_width(m->dims[0], x_dtype, "gnn_train_sample")) return rc;
  if (ld_x < m->dims[0] || (ld_x * (x_dtype == GNN_BF16 ? 2 : 4)) % 16 ||
      (reinterpret_cast<uintptr_t>(X) & 15))
    return fail(GNN_EINVAL, "gnn_train_sample: feature rows must be 16-byte aligned");
  StepPlan p;
  if (int rc = plan_step(m, x_dtype, B, fanouts, csr->num_nodes, ws, ws_bytes, &p, slot)) return rc;
  if (p.bytes > ws_bytes)
    return fail(GNN_EWORKSPACE, "gnn_train_sample: workspace %zu < %zu bytes", ws_bytes, p.bytes);
  hipStream_t st = as_stream(stream);
  // GraphSAGE: the last hop's compaction runs in the layer-1 aggregation
  // launch, which reads the picks (as in gnn_train_step)
  SampleTail tail;
  const bool fuse_tail = m->kind == GNN_SAGE_MEAN;
  if (int rc = sample_blocks_impl(csr, seeds, B, fanouts, m->num_layers, rng_key, p.blocks,
                                  p.sample_ws, p.sample_ws_bytes, nullptr, 0,
                                  fuse_tail ? &tail : nullptr, st, p.tr))
    return rc;
  // layer 1's aggregation needs the blocks and the features only, not the
  // weights: it is part of this call
  const RowSource src{p.layer_blk[0]->src_nodes, csr->num_nodes, ld_x, fuse_tail ? &tail : nullptr};
  return aggregate_layer(p.layer_blk[0], m->kind, X, x_dtype, m->dims[0], p.x[0],
                         x_width(m->kind, m->dims[0], m->dims[1]), src, st,
                         x1_bf16(m, x_dtype) ? GNN_BF16 : GNN_F32);
}

int gnn_train_model(const gnn_model* m, const gnn_csr* csr, const void* X, int32_t x_dtype,
                    int64_t ld_x, const int32_t* labels, const int32_t* seeds, int32_t B,
                    const int32_t* fanouts, float lr, float* loss_out, void* ws, size_t ws_bytes,
                    int32_t slot, void* const* events, void* stream) {
  using namespace gnn;
  if (int rc = check_step_args(m, csr, X, x_dtype, ld_x, labels, seeds, B, loss_out, ws,
                               "gnn_train_model"))
    return rc;
  if (!fanouts) return fail(GNN_EINVAL, "gnn_train_model: null fanouts");
  StepPlan p;
  if (int rc = plan_step(m, x_dtype, B, fanouts, csr->num_nodes, ws, ws_bytes, &p, slot)) return rc;
  if (p.bytes > ws_bytes)
    return fail(GNN_EWORKSPACE, "gnn_train_model: workspace %zu < %zu bytes", ws_bytes, p.bytes);
  hipStream_t st = as_stream(stream);
  const int L = p.L;
  // the first launch (layer-1 aggregation) zeroes the weight gradient and,
  // without the fused output layer, the logits
  FillRange fr[2];
  const int n_fills = step_fills(m, p, fr);
  if (int rc = mark_event(events, GNN_STAGE_SAMPLE, 0, st)) return rc;
  if (int rc = mark_event(events, GNN_STAGE_SAMPLE, 1, st)) return rc;
  return run_model(m, p, X, x_dtype, ld_x, csr->num_nodes, labels, seeds, B, lr, loss_out, events,
                   nullptr, st, fill_pair(fr, n_fills), true);
}

int gnn_train_pipelined(const gnn_model* m, const gnn_csr* csr, const void* X, int32_t x_dtype,
                        int64_t ld_x, const int32_t* labels, const int32_t* const* seeds,
                        const uint64_t* keys, int32_t n, int32_t B, const int32_t* fanouts, float lr,
                        float* loss_out, void* ws, size_t ws_bytes, void* const* events,
                        void* model_stream, void* sample_stream) {
  using namespace gnn;
  if (n < 0 || (n > 0 && (!seeds || !keys || !loss_out)))
    return fail(GNN_EINVAL, "gnn_train_pipelined: bad step arrays");
  // every sampling call keeps its begin launch: skipping it for chained
  // calls (as the workload estimate does) cut 5 us of host time per step but
  // measured 3-4% slower overlapped steps on this schedule
  auto sample = [&](int32_t i, int slot, hipStream_t st) {
    return gnn_train_sample(m, csr, X, x_dtype, ld_x, seeds[i], B, fanouts, keys[i], ws, ws_bytes,
                            slot, st);
  };
  auto model = [&](int32_t i, int slot, hipStream_t st) {
    return gnn_train_model(m, csr, X, x_dtype, ld_x, labels, seeds[i], B, fanouts, lr, loss_out + i,
                           ws, ws_bytes, slot, nullptr, st);
  };
  return gnn::run_pipelined(n, events, as_stream(model_stream), as_stream(sample_stream), sample, model);
}

size_t gnn_shadow_train_workspace_bytes(const gnn_model* m, int32_t x_dtype, int32_t B,
                                        int32_t fanout, int32_t hops) {
  using namespace gnn;
  if (check_model(m, "gnn_shadow_train_workspace_bytes")) return 0;
  StepPlan p;
  if (plan_shadow_step(m, x_dtype, B, fanout, hops, nullptr, 0, &p)) return 0;
  return p.bytes;
}

int gnn_shadow_train_step_views(const gnn_model* m, int32_t x_dtype, int32_t B, int32_t fanout,
                                int32_t hops, void* ws, size_t ws_bytes, gnn_train_views* out) {
  using namespace gnn;
  if (int rc = check_model(m, "gnn_shadow_train_step_views")) return rc;
  if (!ws || !out) return fail(GNN_EINVAL, "gnn_shadow_train_step_views: null pointer");
  StepPlan p;
  if (int rc = plan_shadow_step(m, x_dtype, B, fanout, hops, ws, ws_bytes, &p)) return rc;
  if (p.bytes > ws_bytes) return fail(GNN_EWORKSPACE, "gnn_shadow_train_step_views: workspace too small");
  fill_views(m, p, out);
  return GNN_OK;
}

int gnn_shadow_train_step(const gnn_model* m, const gnn_csr* csr, const void* X, int32_t x_dtype,
                          int64_t ld_x, const int32_t* labels, const int32_t* roots, int32_t B,
                          int32_t fanout, int32_t hops, uint64_t rng_key, float lr, float* loss_out,
                          void* ws, size_t ws_bytes, void* const* events, void* stream) {
  using namespace gnn;
  if (int rc = check_step_args(m, csr, X, x_dtype, ld_x, labels, roots, B, loss_out, ws,
                               "gnn_shadow_train_step"))
    return rc;
  StepPlan p;
  if (int rc = plan_shadow_step(m, x_dtype, B, fanout, hops, ws, ws_bytes, &p)) return rc;
  if (p.bytes > ws_bytes)
    return fail(GNN_EWORKSPACE, "gnn_shadow_train_step: workspace %zu < %zu bytes", ws_bytes, p.bytes);
  hipStream_t st = as_stream(stream);
  const int L = p.L;
  // the layer-1 aggregation launch also zeroes the weight gradient and,
  // without the fused output layer, the logits
  FillRange fr[2];
  const int n_fills = step_fills(m, p, fr);
  if (int rc = mark_event(events, GNN_STAGE_SAMPLE, 0, st)) return rc;
  if (int rc = sample_shadow_impl(csr, roots, B, fanout, hops, rng_key, &p.blocks[0], p.comp_ptr,
                                  p.blocks[1].counts, p.sample_ws, p.sample_ws_bytes, st))
    return rc;
  if (int rc = mark_event(events, GNN_STAGE_SAMPLE, 1, st)) return rc;
  // the roots are local rows 0..B-1
  return run_model(m, p, X, x_dtype, ld_x, csr->num_nodes, labels, roots, B, lr, loss_out, events,
                   nullptr, st, fill_pair(fr, n_fills));
}

int gnn_shadow_train_sample(const gnn_model* m, const gnn_csr* csr, const void* X, int32_t x_dtype,
                            int64_t ld_x, const int32_t* roots, int32_t B, int32_t fanout,
                            int32_t hops, uint64_t rng_key, void* ws, size_t ws_bytes, int32_t slot,
                            void* stream) {
  using namespace gnn;
  if (int rc = check_model(m, "gnn_shadow_train_sample")) return rc;
  if (!csr || !X || !roots || !ws) return fail(GNN_EINVAL, "gnn_shadow_train_sample: null pointer");
  if (B < 1) return fail(GNN_EINVAL, "gnn_shadow_train_sample: empty batch");
  if (x_dtype != GNN_F32 && x_dtype != GNN_BF16) return fail(GNN_EINVAL, "gnn_shadow_train_sample: bad dtype");
  if (int rc = check_width(m->dims[0], x_dtype, "gnn_shadow_train_sample")) return rc;
  if (ld_x < m->dims[0] || (ld_x * (x_dtype == GNN_BF16 ? 2 : 4)) % 16 ||
      (reinterpret_cast<uintptr_t>(X) & 15))
    return fail(GNN_EINVAL, "gnn_shadow_train_sample: feature rows must be 16-byte aligned");
  StepPlan p;
  if (int rc = plan_shadow_step(m, x_dtype, B, fanout, hops, ws, ws_bytes, &p, slot)) return rc;
  if (p.bytes > ws_bytes)
    return fail(GNN_EWORKSPACE, "gnn_shadow_train_sample: workspace %zu < %zu bytes", ws_bytes, p.bytes);
  hipStream_t st = as_stream(stream);
  if (int rc = sample_shadow_impl(csr, roots, B, fanout, hops, rng_key, &p.blocks[0], p.comp_ptr,
                                  p.blocks[1].counts, p.sample_ws, p.sample_ws_bytes, st))
    return rc;
  const RowSource src{p.layer_blk[0]->src_nodes, csr->num_nodes, ld_x};
  return aggregate_layer(p.layer_blk[0], m->kind, X, x_dtype, m->dims[0], p.x[0],
                         x_width(m->kind, m->dims[0], m->dims[1]), src, st,
                         x1_bf16(m, x_dtype) ? GNN_BF16 : GNN_F32);
}

int gnn_shadow_train_model(const gnn_model* m, const gnn_csr* csr, const void* X, int32_t x_dtype,
                           int64_t ld_x, const int32_t* labels, const int32_t* roots, int32_t B,
                           int32_t fanout, int32_t hops, float lr, float* loss_out, void* ws,
                           size_t ws_bytes, int32_t slot, void* const* events, void* stream) {
  using namespace gnn;
  if (int rc = check_step_args(m, csr, X, x_dtype, ld_x, labels, roots, B, loss_out, ws,
                               "gnn_shadow_train_model"))
    return rc;
  StepPlan p;
  if (int rc = plan_shadow_step(m, x_dtype, B, fanout, hops, ws, ws_bytes, &p, slot)) return rc;
  if (p.bytes > ws_bytes)
    return fail(GNN_EWORKSPACE, "gnn_shadow_train_model: workspace %zu < %zu bytes", ws_bytes, p.bytes);
  hipStream_t st = as_stream(stream);
  const int L = p.L;
  FillRange fr[2];
  const int n_fills = step_fills(m, p, fr);
  if (int rc = mark_event(events, GNN_STAGE_SAMPLE, 0, st)) return rc;
  if (int rc = mark_event(events, GNN_STAGE_SAMPLE, 1, st)) return rc;
  return run_model(m, p, X, x_dtype, ld_x, csr->num_nodes, labels, roots, B, lr, loss_out, events,
                   nullptr, st, fill_pair(fr, n_fills), true);
}

int gnn_shadow_train_pipelined(const gnn_model* m, const gnn_csr* csr, const void* X,
                               int32_t x_dtype, int64_t ld_x, const int32_t* labels,
                               const int32_t* const* roots, const uint64_t* keys, int32_t n,
                               int32_t B, int32_t fanout, int32_t hops, float lr, float* loss_out,
                               void* ws, size_t ws_bytes, void* const* events, void* model_stream,
                               void* sample_stream) {
  using namespace gnn;
  if (n < 0 || (n > 0 && (!roots || !keys || !loss_out)))
    return fail(GNN_EINVAL, "gnn_shadow_train_pipelined: bad step arrays");
  auto sample = [&](int32_t i, int slot, hipStream_t st) {
    return gnn_shadow_train_sample(m, csr, X, x_dtype, ld_x, roots[i], B, fanout, hops, keys[i], ws,
                                   ws_bytes, slot, st);
  };
  auto model = [&](int32_t i, int slot, hipStream_t st) {
    return gnn_shadow_train_model(m, csr, X, x_dtype, ld_x, labels, roots[i], B, fanout, hops, lr,
                                  loss_out + i, ws, ws_bytes, slot, nullptr, st);
  };
  return gnn::run_pipelined(n, events, as_stream(model_stream), as_stream(sample_stream), sample, model);
}

}  // extern "C"
