/*
 * gnnhip -- sampling-based mini-batch GNN training on one AMD Instinct MI355X
 * (gfx950).  C ABI.
 *
 * One training step (paper section 2.2, eq. (3)): sample an L-hop
 * computation graph around a batch of seed nodes (Neighbor Sampling: a random
 * selection of every frontier node's neighbours, bounded by a per-hop budget),
 * fetch the features of the sampled nodes, run L message-passing layers
 * (section 2.1: GCN, eq. (1); GraphSAGE, eq. (2)), take the mean loss over
 * the batch, back-propagate and apply an SGD update.
 *
 * Conventions shared by every call
 *  - Pointers are DEVICE pointers (HBM of the current HIP device) unless a
 *    comment says "host".  The caller allocates and owns every buffer; the
 *    library never allocates or frees memory and never synchronises, except
 *    gnn_check_errors.
 *  - `stream` is a hipStream_t passed as void* (NULL = the null stream).  Every
 *    call only enqueues work on it; results are valid once the stream reaches
 *    that point.  Sizes that are only known after sampling (node and edge
 *    counts) stay in device memory (gnn_block.counts) and are never copied
 *    back by the library, so a sequence of calls needs no host round trip.
 *  - Return value: GNN_OK, or a negative code for an error found on the host
 *    before anything was enqueued (nothing is enqueued then).  gnn_last_error()
 *    gives a thread-local message for the last non-zero return.  Errors found
 *    by a kernel (an out-of-range seed, a label outside [0, C), a capacity
 *    overflow) set a sticky per-device error word that gnn_check_errors reports.
 *  - Workspaces of the neighbour sampler (gnn_sample_blocks and the training
 *    steps that include it) keep per-node state between calls.  The first
 *    call on a workspace, or a call with another node count, rebuilds it (one
 *    pass over 8 bytes per node); later calls reuse it.  Between calls its
 *    contents belong to the library, and two calls that may overlap must not
 *    share one workspace.
 *  - Indices are int32 (node ids < 2^31); CSR row pointers are int32 or int64.
 *  - Dense matrices are row-major with a row stride in elements ("ld").
 *  - Feature dtypes: GNN_F32 (float) or GNN_BF16 (bfloat16 bit patterns in
 *    uint16).  All arithmetic accumulates in fp32.
 */
#ifndef GNNHIP_H
#define GNNHIP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  GNN_OK = 0,
  GNN_EINVAL = -1,      /* invalid argument (null pointer, bad size, bad enum) */
  GNN_EWORKSPACE = -2,  /* workspace or a capacity is too small */
  GNN_EHIP = -3,        /* a HIP runtime call or kernel launch failed */
  GNN_EDEVICE = -4      /* (gnn_check_errors only) a kernel flagged bad input */
};

enum { GNN_F32 = 0, GNN_BF16 = 1 };
enum { GNN_SAGE_MEAN = 0, GNN_GCN = 1, GNN_GIN = 2, GNN_GAT = 3 };

/* Device error bits reported by gnn_check_errors through *bits. */
enum {
  GNN_DEVERR_SEED_RANGE = 1,   /* a seed / root id outside [0, num_nodes) */
  GNN_DEVERR_LABEL_RANGE = 2,  /* a label outside [0, num_classes) */
  GNN_DEVERR_CAPACITY = 4,     /* a device-side count exceeded its capacity */
  GNN_DEVERR_GRAPH = 8,        /* a CSR neighbour id outside [0, num_nodes) */
  GNN_DEVERR_SYNC = 16         /* a bounded wait between workgroups of one launch gave up */
};

#define GNN_MAX_LAYERS 4
#define GNN_MAX_FANOUT 64

/* Graph G = (V, E) as CSR (section 2.1): the neighbours N(v) of node v are
 * col[rowptr[v] .. rowptr[v+1]).  The graph must be simple and undirected as
 * the paper's adjacency matrix is (A symmetric, 0/1): every row sorted
 * ascending, no duplicates, no self loops.  The library reads it only. */
typedef struct {
  int64_t num_nodes;
  int64_t num_edges;     /* directed entries = rowptr[num_nodes] */
  const void* rowptr;    /* [num_nodes + 1], int32 or int64 (rowptr_bits) */
  int32_t rowptr_bits;   /* 32 or 64 */
  const int32_t* col;    /* [num_edges] */
  /* Schedule options of the calls that read this graph (zero: the defaults;
   * no result depends on them, they select a schedule, and they let tests
   * exercise every one on small inputs).  scan_order: how the sampler's
   * single-pass scans order their tiles, 0 by block id when the scan grid
   * fits the GPU at once (every tile then waits only on tiles already
   * running) and by tickets taken on arrival otherwise, 1 always by tickets.
   * hub_degree: the degree above which ShaDow's extraction searches a
   * subgraph node's row instead of reading it whole (0: 1024).  Other values
   * (scan_order not 0 or 1, hub_degree < 0) are GNN_EINVAL. */
  int32_t scan_order;
  int32_t hub_degree;
} gnn_csr;

/* One sampled hop: a bipartite block from the dst nodes (the previous
 * frontier, in order) to the src nodes (the next frontier).  The dst nodes are
 * the first n_dst entries of src_nodes.  Edge e of dst row i is
 * indices[indptr[i] + ...], a LOCAL src id; the neighbour's node id is
 * src_nodes[indices[e]].  All arrays are caller-allocated with the capacities
 * below (gnn_block_caps); the library writes them. */
typedef struct {
  int32_t* indptr;     /* [cap_dst + 1] */
  int32_t* indices;    /* [cap_edges] */
  int32_t* src_nodes;  /* [cap_src] node ids, first-occurrence order */
  int32_t* src_occ;    /* [cap_src] times the src node occurs in (dst list ++ edge
                          list): the GCN out-degree with the self edge */
  int32_t* counts;     /* [4] device: n_dst, n_src, n_edges, 0 */
  int32_t cap_dst;
  int32_t cap_src;
  int64_t cap_edges;
} gnn_block;

enum { GNN_OPT_SGD = 0, GNN_OPT_ADAM = 1 };

/* Update rule of the training steps, with g a parameter's gradient of the
 * batch-mean loss and lr the step call's learning rate:
 *   SGD (section 2.2, eq. (3); the default):  w -= lr * g
 *   Adam (the optimiser of the paper's training listings, as defined by
 *   Kingma and Ba, Algorithm 1), step t = ++steps:
 *     m = beta1 m + (1 - beta1) g;  v = beta2 v + (1 - beta2) g^2;
 *     w -= lr * (m / (1 - beta1^t)) / (sqrt(v / (1 - beta2^t)) + eps)
 * computed in fp32, with 1 - beta and the bias corrections rounded to fp32
 * from double. */
typedef struct {
  int32_t kind;      /* GNN_OPT_SGD or GNN_OPT_ADAM */
  double beta1;      /* in [0, 1) */
  double beta2;      /* in [0, 1) */
  double eps;        /* > 0 */
  float* m;          /* Adam: device [gnn_num_params], zero before the first step */
  float* v;          /* Adam: device [gnn_num_params], zero before the first step */
  int64_t steps;     /* Adam steps taken; every training step call adds 1 as it
                        enqueues its update (the steps run in enqueue order) */
} gnn_optimizer;

/* A model of L layers (GraphSAGE-mean, GCN, GIN-0 or one-head GAT, no bias).
 * dims[0] is the input feature width, dims[L] the number of classes.
 * Parameters are one contiguous fp32 buffer: for l = 1..L, GraphSAGE stores
 * W_self (eq. (2) W1) then W_neigh (W2), GCN stores W (eq. (1)), each
 * [dims[l-1] x dims[l]].  GIN and GAT are message-passing models section 2.1
 * names, taken from their own papers:
 *   GIN (Xu et al., ICLR 2019, eq. 4.1, eps = 0): H_l = sigma(relu(Agg W_a) W_b),
 *     Agg = own row + sum of the sampled neighbours; stores W_a [dims[l-1] x
 *     dims[l]] then W_b [dims[l] x dims[l]];
 *   GAT (Velickovic et al., ICLR 2018, eqs. 1-4, one head): T = H W, score
 *     e_vu = LeakyReLU_0.2(a_l . T_v + a_r . T_u) over v's sampled neighbours
 *     and v itself, softmax per row, H_l = sigma(sum_u alpha_vu T_u); stores W
 *     [dims[l-1] x dims[l]] then a_l and a_r (dims[l] each).
 * sigma is ReLU on layers < L.  All row-major.  gnn_train_step updates the
 * buffer in place. */
typedef struct {
  int32_t kind;              /* GNN_SAGE_MEAN, GNN_GCN, GNN_GIN or GNN_GAT */
  int32_t num_layers;        /* 1..GNN_MAX_LAYERS */
  int32_t dims[GNN_MAX_LAYERS + 1];
  float* weights;            /* gnn_num_params() floats */
  gnn_optimizer* opt;        /* NULL: SGD; else the update rule and its state */
} gnn_model;

/* Number of fp32 parameters of the model (host, no device work). */
int64_t gnn_num_params(const gnn_model* m);

/* Upper bounds for the blocks of a batch of B seeds with per-hop budgets
 * fanouts[0..L-1] (hop order: fanouts[0] applies to the seeds) on a graph of
 * N nodes: cap_dst[0] = B, cap_edges[h] = cap_dst[h] * fanouts[h],
 * cap_src[h] = min(N, cap_dst[h] + cap_edges[h]), cap_dst[h+1] = cap_src[h].
 * All outputs are host arrays of L entries.  Returns GNN_EINVAL when L is not
 * in [1, 4], a fanout is not in [1, 64], B < 0 or a bound overflows int32. */
int gnn_block_caps(int32_t B, const int32_t* fanouts /*host*/, int32_t L, int64_t N,
                   int32_t* cap_dst /*host[L]*/, int32_t* cap_src /*host[L]*/,
                   int64_t* cap_edges /*host[L]*/);

/* Scratch bytes gnn_sample_blocks needs for these sizes (16 bytes per graph
 * node of state kept between calls, see the conventions above, plus per-call
 * space). */
size_t gnn_sample_workspace_bytes(int32_t B, const int32_t* fanouts /*host*/, int32_t L, int64_t N);

/* Neighbour sampling of an L-hop computation graph (section 2.2, Neighbor
 * Sampling; budgets of section 5.1.2).  For hop h = 1..L and every dst node v
 * of block h, with d = deg(v) and k = min(fanouts[h-1], d): if d <= k all
 * neighbours are kept, otherwise k distinct CSR positions are drawn with
 * Floyd's algorithm, draw s being word (s mod 4) of Philox4x64-10 at counter
 * (1 + s/4, v, h, 0) under key (rng_key, 0), mapped to [0, m) as
 * floor(r * m / 2^64).  Chosen neighbours are listed in ascending CSR
 * position.  The block's src list is its dst list followed by every other
 * sampled node in first-occurrence order over the edges in (dst, position)
 * order; the next hop's dst list is that src list.  The result depends only
 * on (graph, seeds, fanouts, rng_key): it is bit-for-bit reproducible.
 *
 * seeds: [B] distinct node ids (device).  blocks: host array of L block
 * descriptors (hop order) with capacities >= gnn_block_caps.  ws: device
 * scratch of ws_bytes >= gnn_sample_workspace_bytes (state kept between
 * calls, see the conventions above).  Seeds outside [0, N) raise
 * GNN_DEVERR_SEED_RANGE (their rows are sampled as empty); a CSR neighbour id
 * outside [0, N) raises GNN_DEVERR_GRAPH (the edge then points at local
 * row 0).
 * Errors: GNN_EINVAL (null pointers, L or a fanout out of range, bad
 * rowptr_bits), GNN_EWORKSPACE (a capacity or ws_bytes too small). */
int gnn_sample_blocks(const gnn_csr* csr, const int32_t* seeds, int32_t B,
                      const int32_t* fanouts /*host*/, int32_t L, uint64_t rng_key,
                      gnn_block* blocks /*host[L]*/, void* ws, size_t ws_bytes, void* stream);

/* Feature fetch ("data fetching", section 2.2): out[i, :] = X[ids[i], :] for
 * i < *n_ids.  X: [n_rows x F] with row stride ld_x elements; out: [cap x F]
 * with row stride ld_out.  dtype GNN_F32 or GNN_BF16 (copied bit-exactly).
 * Rows and strides must be 16-byte multiples and both pointers 16-byte
 * aligned.  n_ids: device int32 count (<= cap; a larger count raises
 * GNN_DEVERR_CAPACITY and only cap rows are copied).  An id outside
 * [0, n_rows) raises GNN_DEVERR_SEED_RANGE and its output row is zero. */
int gnn_gather_features(const void* X, int32_t dtype, int64_t n_rows, int64_t ld_x, int32_t F,
                        const int32_t* ids, const int32_t* n_ids /*device*/, int32_t cap,
                        void* out, int64_t ld_out, void* stream);

/* Forward of one layer on one block (section 2.1); kinds GNN_SAGE_MEAN,
 * GNN_GCN and GNN_GIN (GAT layers run inside the training steps only; the
 * kind is rejected with GNN_EINVAL here and in gnn_layer_bwd).  H_in: [n_src x F_in]
 * (row stride F_in, dtype in_dtype) -- the previous layer's output, or the
 * gathered features for layer 1.  The aggregation (Ahat H) is
 *   GNN_SAGE_MEAN: agg_v = (1/c_v) sum over v's c_v sampled edges of H_in[u]
 *                  (agg_v = 0 when c_v = 0);
 *   GNN_GCN:       agg_v = sum over u in {sampled neighbours of v} + {v} of
 *                  H_in[u] / sqrt(src_occ[u] * (c_v + 1));
 *   GNN_GIN:       agg_v = H_in[v] + sum over v's sampled edges of H_in[u].
 * It is written, in fp32, as the layer's GEMM input X [n_dst x K_w]:
 *   GNN_SAGE_MEAN: K_w = 2 F_in, X = [H_in[:n_dst] | agg] (the self rows
 *                  widened to fp32 next to the aggregate);
 *   GNN_GCN:       K_w = F_in, X = agg;
 *   GNN_GIN:       X = [agg | M | pad] with M = relu(agg W_a) the MLP's
 *                  hidden rows (kept for the backward pass), row stride
 *                  F_in + F_out rounded up to a multiple of 4; the weights
 *                  have K_w = F_in + F_out rows.
 * W: [K_w x F_out] fp32 row-major -- for GraphSAGE the stacked [W_self;
 * W_neigh] (eq. (2) W1 over W2), i.e. the two matrices stored one after the
 * other, as in gnn_model; for GCN eq. (1)'s W; for GIN [W_a; W_b].  H_out
 * [n_dst x F_out] fp32: Z = X W (GIN: Z = M W_b), H_out = relu ? max(Z, 0) :
 * Z.  F_in must be a multiple of 4 (fp32) or 8 (bf16); F_in, F_out <= 256. */
int gnn_layer_fwd(const gnn_block* blk, int32_t kind, const void* H_in, int32_t in_dtype,
                  int32_t F_in, const float* W, int32_t F_out, int32_t relu, float* X_out,
                  float* H_out, void* stream);

size_t gnn_layer_bwd_workspace_bytes(int32_t cap_dst, int32_t F_in);

/* Backward of one layer.  X: the forward's X_out; W as in gnn_layer_fwd.
 * dZ: [n_dst x F_out] gradient of the loss w.r.t. the layer's pre-activation
 * output.  Writes (overwrites) dW [K_w x F_out] = X^T dZ (for GraphSAGE the
 * stacked [dW_self; dW_neigh]; for GIN [dW_a; dW_b] with dW_b = M^T dZ,
 * dP = (dZ W_b^T) * (M > 0), dW_a = agg^T dP).  If dH_in is not NULL, also
 * writes the gradient w.r.t. the layer input, [n_src x F_in] fp32: dH_in =
 * Ahat^T (dZ W_neigh^T) (+ dZ W_self^T on the first n_dst rows for
 * GraphSAGE; GIN: Ahat^T (dP W_a^T)), a scatter-add over the block's edges;
 * with mask_relu != 0 it is then multiplied by (H_in > 0) -- H_in [n_src x
 * F_in] fp32, the layer input -- which turns it into the previous layer's dZ
 * when H_in = relu(Z_prev).  ws: ws_bytes >= gnn_layer_bwd_workspace_bytes(
 * cap_dst, F_in), for GIN gnn_layer_bwd_workspace_bytes(cap_dst, 2 F_in +
 * F_out + 4) (the hidden rows' gradient is staged there too); needed
 * whenever dH_in is given or the kind is GIN. */
int gnn_layer_bwd(const gnn_block* blk, int32_t kind, int32_t F_in, const float* X,
                  const float* H_in, const float* W, int32_t F_out, const float* dZ, float* dW,
                  float* dH_in, int32_t mask_relu, void* ws, size_t ws_bytes, void* stream);

/* Mean softmax cross-entropy over B rows (section 2.2, eq. (3)).
 * logits [B x C] (row stride C), labels [B] int32 in [0, C).  Writes
 * dlogits [B x C] = (softmax - onehot) / B and *loss_out (device float).
 * ws: gnn_loss_workspace_bytes(B) bytes. */
size_t gnn_loss_workspace_bytes(int32_t B);
int gnn_softmax_xent(const float* logits, const int32_t* labels, int32_t B, int32_t C,
                     float* dlogits, float* loss_out, void* ws, size_t ws_bytes, void* stream);

/* gnn_softmax_xent for callers that cannot allocate device memory or bring a
 * workspace (code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc): the same kernels, with the per-row losses kept in a
 * library-owned device array of GNN_XENT_NOALLOC_MAX_ROWS floats (256 KiB;
 * one per GPU, held until the process ends) instead of `ws`.  The call
 * allocates nothing.  B > GNN_XENT_NOALLOC_MAX_ROWS returns GNN_EINVAL; other
 * arguments and errors as gnn_softmax_xent.  Calls that overlap on one GPU
 * (different streams or threads) share that array and race. */
#define GNN_XENT_NOALLOC_MAX_ROWS 65536
int gnn_softmax_xent_noalloc(const float* logits, const int32_t* labels, int32_t B, int32_t C,
                             float* dlogits, float* loss_out, void* stream);

/* Plain SGD: w[i] -= lr * g[i] for i < n (section 2.2; no momentum). */
int gnn_sgd(float* w, const float* g, int64_t n, float lr, void* stream);

/* Scratch bytes of one gnn_train_step (includes two slots of blocks, the
 * sampler's workspace with its state kept between calls, every activation and
 * gradient).  x_dtype is the feature dtype. */
size_t gnn_train_workspace_bytes(const gnn_model* m, int32_t x_dtype, int32_t B,
                                 const int32_t* fanouts /*host*/, int64_t N);

/* One neighbour-sampled training step, everything on `stream`, no host sync:
 * sample L hops around `seeds` (gnn_sample_blocks) into block slot 0, read the
 * features of the outermost frontier, run layers 1..L where layer l uses the block of hop
 * L+1-l (so layer L produces the seeds' logits) with ReLU on layers < L,
 * softmax cross-entropy against labels[seeds], back-propagate, and update
 * m->weights in place: W -= lr * dW.  X: [N x dims[0]] features, row stride
 * ld_x, dtype x_dtype.  labels: [N] int32.  loss_out: device float, the batch
 * loss before the update. */
int gnn_train_step(const gnn_model* m, const gnn_csr* csr, const void* X, int32_t x_dtype,
                   int64_t ld_x, const int32_t* labels, const int32_t* seeds, int32_t B,
                   const int32_t* fanouts /*host*/, uint64_t rng_key, float lr, float* loss_out,
                   void* ws, size_t ws_bytes, void* stream);

/* Stages of gnn_train_step_ex that can be bracketed by caller-owned HIP
 * events (for timing): events[2 s] is recorded on the stream before stage s
 * and events[2 s + 1] after it. */
enum {
  GNN_STAGE_SAMPLE = 0,    /* all hops: sampling and relabelling */
  GNN_STAGE_GATHER = 1,    /* feature fetch: empty, the training step's layer-1
                              aggregation reads the feature rows in place (GAT:
                              the widening gather of layer 1's input rows) */
  GNN_STAGE_AGG1 = 2,      /* layer-1 aggregation (one kernel; GAT: scores and
                              attention, after GNN_STAGE_GEMM1) */
  GNN_STAGE_GEMM1 = 3,     /* layer-1 dense update (one kernel; GIN: both MLP
                              products; GAT: T = H W) */
  GNN_STAGE_FWD_REST = 4,  /* layers 2..L forward and the loss */
  GNN_STAGE_BACKWARD = 5,  /* every layer's backward */
  GNN_STAGE_SGD = 6,       /* parameter update and loss reduction */
  GNN_NUM_STAGES = 7
};

/* gnn_train_step with optional stage events: `events` is NULL or an array of
 * 2 * GNN_NUM_STAGES hipEvent_t handles (passed as void*) owned by the caller. */
int gnn_train_step_ex(const gnn_model* m, const gnn_csr* csr, const void* X, int32_t x_dtype,
                      int64_t ld_x, const int32_t* labels, const int32_t* seeds, int32_t B,
                      const int32_t* fanouts /*host*/, uint64_t rng_key, float lr, float* loss_out,
                      void* ws, size_t ws_bytes, void* const* events, void* stream);

/* Where gnn_train_step keeps its intermediates inside `ws` (for inspection
 * after the stream has finished): the L blocks (hop order), xg = NULL (the
 * step gathers no feature copy: layer 1 reads the rows of X through its
 * block's src node ids), and per layer l = 1..L (index l-1) the GEMM input X (as in
 * gnn_layer_fwd: [H_dst | agg] for GraphSAGE, agg for GCN, [agg | M] for GIN;
 * row stride x_ld[l] elements, element type x_dtype[l]: GNN_F32, except that
 * a step with bf16 features keeps layer 1's GraphSAGE / GCN input in
 * GNN_BF16, rounded to nearest even -- the operand of that layer's products,
 * which take bf16 operands with fp32 accumulation),
 * the output H_l (post-ReLU; logits for l = L), and the weight gradient of
 * the step (gnn_num_params floats, same layout as the weights).  Host-only. */
typedef struct {
  gnn_block blocks[GNN_MAX_LAYERS];
  void* xg;
  float* x[GNN_MAX_LAYERS];
  int32_t x_ld[GNN_MAX_LAYERS];
  int32_t x_dtype[GNN_MAX_LAYERS];
  float* h[GNN_MAX_LAYERS];
  float* dweights;
  float* dlogits;
  int32_t* comp_ptr;  /* ShaDow only: [B + 1] component offsets (else NULL) */
} gnn_train_views;

int gnn_train_step_views(const gnn_model* m, int32_t x_dtype, int32_t B,
                         const int32_t* fanouts /*host*/, int64_t N, void* ws, size_t ws_bytes,
                         gnn_train_views* out /*host*/);

/* gnn_train_step_views for block slot `slot` (0 or 1) of the two-slot
 * workspace of pipelined steps: the blocks and layer 1's GEMM input x[0] are
 * those of the last batch sampled into that slot; the other fields (layers
 * >= 2, outputs, weight gradient) are shared by the slots and hold the last
 * model pass.  gnn_train_step_views is slot 0.  Errors: as
 * gnn_train_step_views, and GNN_EINVAL for a slot other than 0 or 1. */
int gnn_train_slot_views(const gnn_model* m, int32_t x_dtype, int32_t B,
                         const int32_t* fanouts /*host*/, int64_t N, void* ws, size_t ws_bytes,
                         int32_t slot, gnn_train_views* out /*host*/);

/* A training step in two parts, so that the next batch can be sampled while
 * the current one trains (on two streams).  gnn_train_sample does the
 * sampling of gnn_train_step for `seeds` into block slot `slot` (0 or 1) of
 * the workspace, and layer 1's aggregation of the features X (it needs no
 * weights) into the slot; gnn_train_model then runs the rest of the step
 * (layer 1's product, layers 2..L, loss, backward, SGD) on that slot.  Each call enqueues on
 * its own `stream` and returns at once.  Ordering the caller provides (with
 * events): a model call after the sample call of its slot; a sample call
 * into a slot after the previous model call on that slot has finished;
 * sample calls one after another (they share the sampler's state) and model
 * calls one after another (they share the weights and the model's buffers).
 * gnn_train_step is gnn_train_sample(slot 0) + gnn_train_model(slot 0) on one
 * stream, with the results of those two calls.  Arguments as gnn_train_step;
 * events as gnn_train_step_ex (the sampling stage is recorded empty).
 * Errors: as gnn_train_step, and GNN_EINVAL for a slot other than 0 or 1. */
int gnn_train_sample(const gnn_model* m, const gnn_csr* csr, const void* X, int32_t x_dtype,
                     int64_t ld_x, const int32_t* seeds, int32_t B,
                     const int32_t* fanouts /*host*/, uint64_t rng_key, void* ws, size_t ws_bytes,
                     int32_t slot, void* stream);
int gnn_train_model(const gnn_model* m, const gnn_csr* csr, const void* X, int32_t x_dtype,
                    int64_t ld_x, const int32_t* labels, const int32_t* seeds, int32_t B,
                    const int32_t* fanouts /*host*/, float lr, float* loss_out, void* ws,
                    size_t ws_bytes, int32_t slot, void* const* events, void* stream);

/* n training steps in that overlapped order, enqueued with one call: the
 * sample part of step i + 1 on sample_stream while step i's model part runs
 * on model_stream, slots alternating (step i uses slot i mod 2), the model
 * stream waiting at the end for the sample stream.  seeds: host array of n
 * device pointers (the [B] seeds of each step); keys: host array of n
 * sampling keys; loss_out: device float[n], the loss of step i before its
 * update.  events: host array of 4 hipEvent_t created by the caller (timing
 * may be disabled; they must not be in use elsewhere until the streams have
 * finished).  Other arguments as gnn_train_step.  Returns after enqueueing;
 * on an error part of the steps may have been enqueued. */
int gnn_train_pipelined(const gnn_model* m, const gnn_csr* csr, const void* X, int32_t x_dtype,
                        int64_t ld_x, const int32_t* labels, const int32_t* const* seeds /*host*/,
                        const uint64_t* keys /*host*/, int32_t n, int32_t B,
                        const int32_t* fanouts /*host*/, float lr, float* loss_out, void* ws,
                        size_t ws_bytes, void* const* events /*host[4]*/, void* model_stream,
                        void* sample_stream);

/* ---- ShaDow k-hop subgraphs (section 2.2, ShaDow K-Hop Sampling; section
 * 5.2: ShaDow constructs mini-batches by inducing all edges among a node set
 * sampled around each root) ------------------------------------------------
 *
 * For every root r, hops are taken breadth-first: hop h samples, with the
 * rule and the Philox stream of gnn_sample_blocks (key (rng_key, 0), counter
 * word 2 = h), only the nodes first reached at hop h-1 (hop 1 samples the
 * root); new nodes join the root's set in order of first occurrence.  The
 * subgraph keeps every graph edge between two nodes of the set.  The batch
 * is the disjoint union of the roots' subgraphs as one square block
 * (n_dst == n_src == total nodes): root r has local id r, then each
 * component's other nodes follow, component after component, in
 * first-occurrence order, so the roots' rows are the prefix 0..B-1.  Rows
 * list their induced neighbours in ascending global id.  src_occ[u] =
 * 1 + induced degree of u (the GCN out-degree with the self edge).
 *
 * The graph must be symmetric (each edge stored in both directions, as for an
 * undirected graph) with every CSR row sorted by neighbour id: the induced
 * subgraphs then are symmetric too, so a row's length is also the node's
 * out-degree (src_occ) and the training step's backward gathers over the
 * union block as its own transpose; and the rows of high-degree nodes need
 * not be read whole (an induced edge is found from its lower-degree
 * endpoint's row, or by a binary search between two high-degree rows).
 *
 * Capacities: at most sum_{h=0..hops} fanout^h nodes per root (<= 2048);
 * cap_nodes = B * that, cap_edges = cap_nodes * (that - 1).  hops in [1, 3]. */
int gnn_shadow_caps(int32_t B, int32_t fanout, int32_t hops, int32_t* cap_nodes /*host*/,
                    int64_t* cap_edges /*host*/);
size_t gnn_shadow_workspace_bytes(int32_t B, int32_t fanout, int32_t hops);

/* roots: [B] device node ids.  sub: the union block (cap_dst = cap_src >=
 * cap_nodes, cap_edges as gnn_shadow_caps); sub->counts = {total, total, E,
 * 0}.  comp_ptr: [B + 1] device, component r's non-root nodes are local ids
 * [comp_ptr[r], comp_ptr[r+1]).  readout_counts: device int32[4] = {B,
 * total, edges of the root rows, 0} -- with it, sub's arrays describe the
 * block of the root rows alone (used for the output layer). */
int gnn_sample_shadow(const gnn_csr* csr, const int32_t* roots, int32_t B, int32_t fanout,
                      int32_t hops, uint64_t rng_key, gnn_block* sub, int32_t* comp_ptr,
                      int32_t* readout_counts, void* ws, size_t ws_bytes, void* stream);

/* One ShaDow training step: gnn_sample_shadow around `roots`, gather the
 * features of every node of the union, layers 1..L-1 on the whole union
 * block, layer L on the roots' rows (the readout: a root's prediction is its
 * own row), softmax cross-entropy against labels[roots], backward, SGD.  Other
 * arguments as gnn_train_step_ex. */
size_t gnn_shadow_train_workspace_bytes(const gnn_model* m, int32_t x_dtype, int32_t B,
                                        int32_t fanout, int32_t hops);
int gnn_shadow_train_step(const gnn_model* m, const gnn_csr* csr, const void* X, int32_t x_dtype,
                          int64_t ld_x, const int32_t* labels, const int32_t* roots, int32_t B,
                          int32_t fanout, int32_t hops, uint64_t rng_key, float lr, float* loss_out,
                          void* ws, size_t ws_bytes, void* const* events, void* stream);
/* Views of a ShaDow step: blocks[0] the union block, blocks[1] the root rows,
 * comp_ptr set; other fields as gnn_train_step_views. */
int gnn_shadow_train_step_views(const gnn_model* m, int32_t x_dtype, int32_t B, int32_t fanout,
                                int32_t hops, void* ws, size_t ws_bytes,
                                gnn_train_views* out /*host*/);
/* The two parts of a ShaDow step (subgraph extraction and layer 1's
 * aggregation into block slot `slot`; the rest of the step on that slot),
 * with the ordering rules of gnn_train_sample / gnn_train_model. */
int gnn_shadow_train_sample(const gnn_model* m, const gnn_csr* csr, const void* X, int32_t x_dtype,
                            int64_t ld_x, const int32_t* roots, int32_t B, int32_t fanout,
                            int32_t hops, uint64_t rng_key, void* ws, size_t ws_bytes, int32_t slot,
                            void* stream);
int gnn_shadow_train_model(const gnn_model* m, const gnn_csr* csr, const void* X, int32_t x_dtype,
                           int64_t ld_x, const int32_t* labels, const int32_t* roots, int32_t B,
                           int32_t fanout, int32_t hops, float lr, float* loss_out, void* ws,
                           size_t ws_bytes, int32_t slot, void* const* events, void* stream);
/* n ShaDow steps overlapped as gnn_train_pipelined (roots: host array of n
 * device pointers). */
int gnn_shadow_train_pipelined(const gnn_model* m, const gnn_csr* csr, const void* X,
                               int32_t x_dtype, int64_t ld_x, const int32_t* labels,
                               const int32_t* const* roots /*host*/, const uint64_t* keys /*host*/,
                               int32_t n, int32_t B, int32_t fanout, int32_t hops, float lr,
                               float* loss_out, void* ws, size_t ws_bytes,
                               void* const* events /*host[4]*/, void* model_stream,
                               void* sample_stream);

/* ---- Dynamic load balancing (section 3, Dynamic Load Balancer: before
 * training, the sampling algorithm runs on every mini-batch and the
 * aggregations of its computation graph are counted; batches are then handed
 * to workers by that estimated workload in proportion to the workers' speeds,
 * and the proportion is re-derived from measured times after an epoch) ----- */

/* Workload estimate of n neighbour-sampled mini-batches for model m (only
 * m->kind, num_layers and dims are read; weights may be NULL).  Batch i is
 * sampled as the training step samples it (seeds[i], keys[i], fanouts: the
 * same blocks, see gnn_sample_blocks), and
 *   work[i] = sum over layers l of (E_l + [GCN, GIN] n_dst_l) * dims[l - 1],
 * the feature-element additions of the layers' aggregations: layer l runs on
 * the block of hop L + 1 - l, E_l is that block's sampled edge count and
 * n_dst_l its dst row count (GCN's normalised adjacency and GIN's sum also
 * add each row's own features).  edges: NULL or device int64[n * L], E of hop h + 1 of batch
 * i at [i * L + h].  seeds: host array of n device pointers to B distinct node
 * ids each; keys: host[n].  work: device int64[n].  ws: ws_bytes >=
 * gnn_estimate_workspace_bytes(B, fanouts, L, N) (a block set and the
 * sampler's scratch, with the per-node state rules of gnn_sample_blocks).
 * Errors: GNN_EINVAL (null pointers, bad model, n < 0, B < 1),
 * GNN_EWORKSPACE; device errors as gnn_sample_blocks. */
size_t gnn_estimate_workspace_bytes(int32_t B, const int32_t* fanouts /*host*/, int32_t L,
                                    int64_t N);
int gnn_estimate_work(const gnn_model* m, const gnn_csr* csr, const int32_t* const* seeds /*host*/,
                      const uint64_t* keys /*host*/, int32_t n, int32_t B,
                      const int32_t* fanouts /*host*/, int64_t* work, int64_t* edges, void* ws,
                      size_t ws_bytes, void* stream);

/* The same for ShaDow mini-batches (gnn_sample_shadow around roots[i] with
 * keys[i]): layers 1..L-1 run on the union block and layer L on the roots'
 * rows, so work[i] = sum over l < L of (E + [GCN, GIN] n) * dims[l - 1] +
 * (E_roots + [GCN, GIN] B) * dims[L - 1], with n the union's node count, E its
 * edges and E_roots the edges of the roots' rows.  edges: NULL or device
 * int64[n * 2] = (E, E_roots) per batch.  ws_bytes >=
 * gnn_shadow_estimate_workspace_bytes(B, fanout, hops). */
size_t gnn_shadow_estimate_workspace_bytes(int32_t B, int32_t fanout, int32_t hops);
int gnn_shadow_estimate_work(const gnn_model* m, const gnn_csr* csr,
                             const int32_t* const* roots /*host*/, const uint64_t* keys /*host*/,
                             int32_t n, int32_t B, int32_t fanout, int32_t hops, int64_t* work,
                             int64_t* edges, void* ws, size_t ws_bytes, void* stream);

/* Assignment of n batches to k workers by estimated workload (host only, no
 * GPU work).  Worker j's target is ratio[j] / sum(ratio) of the total
 * workload; batches are taken heaviest first (ties: lower index) and each
 * goes to the worker whose assigned workload lies furthest below its target
 * (ties: lower worker id).  No worker ends more than one batch's workload
 * above its target.  work: host[n], each >= 0; ratio: host[k], finite, >= 0,
 * positive sum; worker: host[n] receives worker ids; load: NULL or host[k]
 * receives each worker's summed workload.  Errors: GNN_EINVAL. */
int gnn_dlb_assign(const int64_t* work /*host*/, int32_t n, const double* ratio /*host*/, int32_t k,
                   int32_t* worker /*host*/, int64_t* load /*host, may be NULL*/);

/* The next epoch's ratio from the last one's measurement (host only).
 * Worker j processed load[j] units of workload in seconds[j]; its speed is
 * load[j] / seconds[j].  Workers with load and time are measured; if their
 * times differ by more than tolerance * (the largest time), each measured
 * worker's new ratio is its speed's share of the measured workers' summed
 * speed, times the previous share those workers held together; workers
 * without a measurement, or balanced times, keep the previous ratio (all
 * normalised to sum 1).  Errors: GNN_EINVAL (negative or non-finite entries,
 * prev summing to 0, tolerance < 0). */
int gnn_dlb_ratio(const int64_t* load /*host*/, const double* seconds /*host*/,
                  const double* prev /*host*/, int32_t k, double tolerance,
                  double* ratio /*host*/);

/* ---- GPU feature caching (section 3, GPU Feature Caching: the feature
 * table stays in host memory, rows the GPU needs are read over the host link,
 * and least-recently-used replacement keeps a set of rows in GPU memory so
 * that frequently needed rows cross the link once) ------------------------
 *
 * The cache is set-associative: node v lives in set fmix32(v) mod num_sets
 * (fmix32: MurmurHash3's 32-bit finaliser), in one of `ways` entries.
 * Recency is counted in fetch calls: call t (1, 2, ... since the last reset)
 * stamps every entry it reads with t.  After its lookups, each set takes in
 * its missed nodes in request order for as long as it has entries not read
 * by this call, replacing them oldest stamp first (never-used entries
 * first; ties: lower way); further misses are served without being cached.
 * All choices are deterministic. */
typedef struct {
  int32_t num_sets;  /* >= 1 */
  int32_t ways;      /* 1..64 */
  int32_t width;     /* row elements; width * element size a multiple of 16 bytes */
  int32_t dtype;     /* GNN_F32 or GNN_BF16 */
  void* mem;         /* device, 256-byte aligned, gnn_feature_cache_bytes bytes;
                        owned by the caller, contents owned by the library */
} gnn_feature_cache;

/* Bytes of cache memory (0 for invalid sizes): the entries' keys, stamps and
 * rows (num_sets * ways rows) plus per-set counters. */
size_t gnn_feature_cache_bytes(int32_t num_sets, int32_t ways, int32_t width, int32_t dtype);
/* Empties the cache (every call starts from this state). */
int gnn_feature_cache_reset(const gnn_feature_cache* c, void* stream);
/* Device addresses of the cache's entries (host arithmetic only, no GPU
 * work): keys [num_sets * ways] int32 (-1 = empty; entry e = set * ways +
 * way), stamps [num_sets * ways] uint32 (0 = never used) and rows
 * [num_sets * ways] of width elements each, contiguous.  Any may be NULL. */
int gnn_feature_cache_views(const gnn_feature_cache* c, int32_t** keys, uint32_t** stamps,
                            void** rows);

/* out[i] = X[ids[i]] for i < min(*n_ids, cap) (ids: device; the count is read
 * on the device and a count above cap raises GNN_DEVERR_CAPACITY), each row
 * served from the cache when present and read from X otherwise; then the
 * replacement step above.  X: [n_rows x ld_x] of the cache's dtype, in memory
 * the device can read (host memory allocated pinned and mapped, e.g. by
 * hipHostMalloc, or device memory), 16-byte aligned rows.  out: device
 * [cap x ld_out].  The ids of one call must be distinct (a block's node list
 * is).  An id outside [0, n_rows) raises GNN_DEVERR_SEED_RANGE, gives a zero
 * row and is not cached.  stats: device uint64[2] += (hits, misses).  ws:
 * ws_bytes >= gnn_gather_cached_workspace_bytes(num_sets, cap).  Calls that
 * use one cache must not overlap.  Errors: GNN_EINVAL, GNN_EWORKSPACE. */
size_t gnn_gather_cached_workspace_bytes(int32_t num_sets, int32_t cap);
int gnn_gather_cached(const gnn_feature_cache* c, const void* X, int64_t n_rows, int64_t ld_x,
                      const int32_t* ids, const int32_t* n_ids, int32_t cap, void* out,
                      int64_t ld_out, uint64_t* stats, void* ws, size_t ws_bytes, void* stream);

/* A training step whose feature table stays in host memory (section 3: the
 * features of large graphs are kept in host memory and fetched over the host
 * link, with GPU feature caching of the frequently needed rows).  As
 * gnn_train_step, except that after sampling the feature rows of the last
 * hop's src nodes are fetched through `cache` (gnn_gather_cached; X: device-
 * readable host memory as described there, cache rows of x_dtype and width
 * dims[0]) into the workspace, and layer 1 reads that copy.  cache_stats:
 * device uint64[2] += (hits, misses).  ws_bytes >=
 * gnn_train_cached_workspace_bytes(m, x_dtype, B, fanouts, N,
 * cache->num_sets); the workspace starts with the layout of
 * gnn_train_step_views. */
size_t gnn_train_cached_workspace_bytes(const gnn_model* m, int32_t x_dtype, int32_t B,
                                        const int32_t* fanouts /*host*/, int64_t N,
                                        int32_t num_sets);
int gnn_train_step_cached(const gnn_model* m, const gnn_csr* csr, const void* X, int32_t x_dtype,
                          int64_t ld_x, const gnn_feature_cache* cache, uint64_t* cache_stats,
                          const int32_t* labels, const int32_t* seeds, int32_t B,
                          const int32_t* fanouts /*host*/, uint64_t rng_key, float lr,
                          float* loss_out, void* ws, size_t ws_bytes, void* stream);

/* Waits for `stream`, then returns GNN_EDEVICE and the device error bits
 * (GNN_DEVERR_*) in *bits if any kernel flagged an error since the last call
 * (and clears them), GNN_OK otherwise, or GNN_EHIP on a HIP failure. */
int gnn_check_errors(void* stream, int32_t* bits /*host, may be NULL*/);

/* Thread-local message of the last non-zero return on this thread. */
const char* gnn_last_error(void);

/* Library version string. */
const char* gnn_version(void);

/* Launch tracing, a timing aid.  While a trace is installed on the calling
 * thread, every kernel the library enqueues from that thread is launched with
 * two caller-created HIP events that take the kernel's own start and end
 * timestamps (hipExtLaunchKernel): the i-th recorded launch uses events[2 i]
 * and events[2 i + 1], and names[i] receives the kernel's static name:
 * "begin", "sample", "scans", "indices" (neighbour sampling), "shadow_build",
 * "shadow_scan", "shadow_emit" (ShaDow), "gather", "aggregate", "gemm_fwd",
 * "gemm_dw", "gemm_dx", "scatter", "relu_mask", "softmax_xent", "sgd",
 * "fill", "head", "work" (workload estimate), "cache_lookup", "cache_scan",
 * "cache_place", "cache_insert" (feature cache), "gat_scores", "gat_attend",
 * "gat_attend_bwd", "gat_score_grad", "gat_colsum", "gat_colsum_final" (GAT).
 * In a training step some launches carry neighbouring work: "begin"
 * also zeroes the gradient buffers, "gather" also compacts the last hop's
 * edges, "gemm_dx" also zeroes the rows the scatter adds into, and the GEMMs
 * read dZ through the ReLU mask (no "relu_mask" launch).  With `only` set, other kernels are not recorded.  A launch beyond
 * `capacity`, or without a pair of events, is counted in `dropped` instead. */
typedef struct {
  void* const* events;  /* [2 * capacity] hipEvent_t, created by the caller */
  const char** names;   /* [capacity] host array, or NULL */
  const char* only;     /* record only this kernel name, or NULL for all */
  int32_t capacity;
  int32_t count;        /* recorded launches (updated by the library) */
  int32_t dropped;      /* launches not recorded (updated by the library) */
} gnn_trace;

/* Installs `t` for the calling thread (NULL removes it).  The struct must
 * stay valid while it is installed.  Errors: GNN_EINVAL (capacity < 0, or
 * capacity > 0 without events). */
int gnn_trace_begin(gnn_trace* t);

#ifdef __cplusplus
}
#endif
#endif /* GNNHIP_H */
