// Internal declarations shared by the translation units of libgnnhip.so.
// Each .hip file owns its kernels and exposes host-side launchers declared
// here; no kernel is launched across translation units.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

#include "../../include/gnnhip.h"
#include "relabel.hpp"

namespace gnn {

// ---- errors ---------------------------------------------------------------
int fail(int code, const char* fmt, ...);
int hip_fail(hipError_t e, const char* what);
#define GNN_HIP_TRY(call)                                   \
  do {                                                      \
    hipError_t e_ = (call);                                 \
    if (e_ != hipSuccess) return ::gnn::hip_fail(e_, #call); \
  } while (0)
#define GNN_LAUNCH_CHECK(what)                                         \
  do {                                                                 \
    hipError_t e_ = hipGetLastError();                                 \
    if (e_ != hipSuccess) return ::gnn::hip_fail(e_, what);            \
  } while (0)

// ---- launches and tracing (common.hip) ----------------------------------------
// If the calling thread's installed gnn_trace records launches of `name`,
// takes its next pair of events (kernel start and end) and returns true.
bool trace_slot(const char* name, hipEvent_t* start, hipEvent_t* stop);

// kernel<<<grid, block, shmem, st>>>(args...); a traced launch carries the
// trace's events, which take the kernel's own start and end timestamps.
template <typename... Formals, typename... Args>
inline void launch(const char* name, void (*kernel)(Formals...), dim3 grid, dim3 block,
                   uint32_t shmem, hipStream_t st, Args... args) {
  hipEvent_t start = nullptr, stop = nullptr;
  trace_slot(name, &start, &stop);
  hipExtLaunchKernelGGL(kernel, grid, block, shmem, st, start, stop, 0u, args...);
}

// Sticky device error word of the current device (bits GNN_DEVERR_*).
int* device_error_word();

// Compute units of the current device (cached per device).
int device_cu_count();

inline hipStream_t as_stream(void* s) { return reinterpret_cast<hipStream_t>(s); }

// ---- workspace carving ------------------------------------------------------
struct Carver {
  char* base;
  size_t off = 0;
  size_t cap;
  explicit Carver(void* b, size_t c) : base(static_cast<char*>(b)), cap(c) {}
  template <typename T>
  T* take(size_t n) {
    off = (off + 255) & ~size_t(255);
    T* p = base ? reinterpret_cast<T*>(base + off) : nullptr;
    off += n * sizeof(T);
    return p;
  }
  bool fits() const { return off <= cap; }
};

inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// the schedule options of a graph (scan_order 0 or 1, hub_degree >= 0)
inline int check_csr_options(const gnn_csr* csr, const char* who) {
  if (csr->scan_order != 0 && csr->scan_order != 1)
    return fail(GNN_EINVAL, "%s: scan_order %d not 0 or 1", who, csr->scan_order);
  if (csr->hub_degree < 0) return fail(GNN_EINVAL, "%s: hub_degree %d < 0", who, csr->hub_degree);
  return GNN_OK;
}

// ---- fill (common.hip) --------------------------------------------------------
struct FillRange {
  void* p;
  int64_t n_words;  // 32-bit words
  int32_t value;
};
int launch_fill(const FillRange* ranges, int n, hipStream_t st);  // n <= 8

// Up to two fill ranges carried by another launch as extra blocks.
struct FillPair {
  int32_t* p[2] = {nullptr, nullptr};
  int64_t n[2] = {0, 0};
  int32_t v[2] = {0, 0};
};
inline FillPair fill_pair(const FillRange* r, int n) {
  FillPair f;
  for (int i = 0; i < n && i < 2; ++i) {
    f.p[i] = static_cast<int32_t*>(r[i].p);
    f.n[i] = r[i].p ? r[i].n_words : 0;
    f.v[i] = r[i].value;
  }
  return f;
}
// fill blocks such a launch appends: 0 if there is nothing to fill
inline int64_t fill_blocks(const FillPair& f, int threads) {
  const int64_t mx = f.n[0] > f.n[1] ? f.n[0] : f.n[1];
  if (mx <= 0) return 0;
  const int64_t b = ceil_div(mx, (int64_t)threads * 4);
  return b > 512 ? 512 : b;
}
__device__ __forceinline__ void run_fills(const FillPair& f, int64_t block, int64_t blocks, int threads) {
  const int64_t stride = blocks * threads;
  for (int r = 0; r < 2; ++r)
    for (int64_t i = block * threads + threadIdx.x; i < f.n[r]; i += stride) f.p[r][i] = f.v[r];
}

// ---- sampling (sample.hip) --------------------------------------------------
size_t sample_scratch_bytes(const int32_t* cap_dst, const int32_t* cap_src,
                            const int64_t* cap_edges, int32_t L, int64_t N);
// extra: up to 4 fill ranges done by the sampler's first launch.  tail: if not
// null, the last hop's edge compaction is not launched but returned, for the
// caller's next launch to run (finish_sampling); the blocks are complete only
// after it.
// Transpose buffers of one block (src -> dst lists), see TransposeJob.
struct BlockTranspose {
  int32_t* t_ptr = nullptr;  // [cap_src + 1]
  int32_t* t_cur = nullptr;  // [cap_src]
  int32_t* t_dst = nullptr;  // [cap_edges]
};
// tr (optional): per hop h < L - 1 with t_ptr set, the call also builds the
// block's transpose (complete with the call, like the block itself).
// chained: the previous call on this scratch (same sizes, same stream order)
// was a sampling call whose last step prepared this one, and fewer than
// kChainCalls calls have been chained since a call that was not; the begin
// launch is then skipped (unless there are fills to do).
int sample_blocks_impl(const gnn_csr* csr, const int32_t* seeds, int32_t B,
                       const int32_t* fanouts, int32_t L, uint64_t rng_key, gnn_block* blocks,
                       void* ws, size_t ws_bytes, const FillRange* extra, int n_extra,
                       SampleTail* tail, hipStream_t st, const BlockTranspose* tr = nullptr,
                       bool chained = false);

// ---- ShaDow (shadow.hip) ------------------------------------------------------
int shadow_caps(int32_t B, int32_t fanout, int32_t hops, int32_t* cap_nodes, int64_t* cap_edges);
size_t shadow_scratch_bytes(int32_t B, int32_t fanout, int32_t hops);
int sample_shadow_impl(const gnn_csr* csr, const int32_t* roots, int32_t B, int32_t fanout,
                       int32_t hops, uint64_t rng_key, gnn_block* sub, int32_t* comp_ptr,
                       int32_t* readout_counts, void* ws, size_t ws_bytes, hipStream_t st);

// ---- gather (gather.hip) ----------------------------------------------------
// tail (optional): a sampling call's last step, run by extra blocks.
int launch_gather(const void* X, int32_t esize, int64_t n_rows, int64_t ld_x, int32_t F,
                  const int32_t* ids, const int32_t* n_ids, int32_t cap, void* out, int64_t ld_out,
                  const SampleTail* tail, hipStream_t st);

// ---- aggregation (aggregate.hip) ----------------------------------------------
// Rows v < counts[0] of the layer's GEMM input X (row stride out_ld):
// SAGE: X[v] = [H[v] | agg_v] (out_ld >= 2F); GCN: X[v] = agg_v, where
// agg_v = sum_e w_e H[idx_e] (+ GCN self term).  Local row u of H is H row u
// (stride F), or, if `rows` is given, H row rows[u] (stride ld_h elements,
// a 16-byte multiple; rows outside [0, n_rows) read as zeros).
// `fills`: done by extra blocks of the same launch.  out_dtype: X in fp32, or
// in bf16 rounded to nearest even (bf16 input rows, SAGE or GCN).
int launch_aggregate(const gnn_block* blk, int32_t kind, const void* H, int32_t dtype, int32_t F,
                     void* out, int32_t out_ld, hipStream_t st, const int32_t* rows = nullptr,
                     int64_t n_rows = 0, int64_t ld_h = 0, const FillPair& fills = FillPair{},
                     int32_t out_dtype = GNN_F32);
// GraphSAGE-mean layer input of the last sampled hop's block `blk` (its
// src_nodes and capacity) from the hop's padded picks held by a sampling
// call's `tail`, reading rows of the feature table H (n_rows rows, stride
// ld_h); the same launch finishes the sampling call (the block's edge
// compaction).
struct WtJob;
int launch_aggregate_picks(const SampleTail& tail, const gnn_block* blk, const void* H,
                           int32_t dtype, int32_t F, int64_t n_rows, int64_t ld_h, void* out,
                           int32_t out_ld, hipStream_t st, int32_t out_dtype = GNN_F32,
                           const WtJob* wt = nullptr);
// dH[idx_e] += w_e dAgg[v] (+ GCN self edge) with fp32 atomics.
int launch_scatter(const gnn_block* blk, int32_t kind, const float* dAgg, int32_t F, float* dH,
                   hipStream_t st);
// The same backward as a gather over the block's transpose (t_ptr, t_dst):
// every row u < n_src of dH is written once; SAGE rows u < n_dst must already
// hold the self path (they are added to).  F a multiple of 4, at most 256.
// With mask ([n_src x F] fp32; SAGE or GCN) every row is written times
// (mask > 0): to dH, or with out16 to out16 instead, as bf16 (nearest even).
int launch_scatter_t(const gnn_block* blk, int32_t kind, const int32_t* t_ptr, const int32_t* t_dst,
                     const float* dAgg, int32_t F, float* dH, hipStream_t st,
                     const float* mask = nullptr, uint16_t* out16 = nullptr);
// x[i] *= (h[i] > 0) over rows < counts[1] (src count) of a [rows x F] matrix.
int launch_relu_mask(const gnn_block* blk, const float* h, int32_t F, float* x, hipStream_t st);

// GAT layer (gat.hip).  T rows have stride ldt (F rounded up to 4); s holds
// (a_l . T_u, a_r . T_u) per src row u, stats (m_v, 1 / normaliser) per dst
// row v; a = [a_l; a_r] (2 x F).
int launch_gat_gather(const gnn_block* blk, const void* X, int32_t dtype, const int32_t* rows,
                      int64_t n_rows, int64_t ld_x, int32_t F, float* out, hipStream_t st);
int launch_gat_scores(const gnn_block* blk, const float* T, int32_t ldt, const float* a, int32_t F,
                      float* s, hipStream_t st);
int launch_gat_attend(const gnn_block* blk, const float* T, int32_t ldt, const float* s, int32_t F,
                      int32_t relu, float* out, float* stats, hipStream_t st);
int launch_gat_attend_bwd(const gnn_block* blk, const float* T, int32_t ldt, const float* s,
                          const float* stats, const float* dout, int64_t ld_do, const float* mask,
                          int32_t F, float* dT, float* ds, hipStream_t st);
int launch_gat_score_grad(const gnn_block* blk, const float* a, int32_t F, const float* ds, float* dT,
                          int32_t ldt, hipStream_t st);
// out[c * oc + f * of] = sum over rows u < min(*n_dev, cap) of w[2u + c] X[u, f]
// (c = 0, 1; f < F; X row stride ld), the [ds_l | ds_r]^T X products, in a
// fixed order through `part` (gat_colsum_part_floats() floats).
size_t gat_colsum_part_floats();
int launch_gat_colsum2(const int32_t* n_dev, int32_t cap, const float* w, const float* X, int64_t ld,
                       int32_t F, float* part, float* out, int64_t oc, int64_t of, hipStream_t st);

// ---- GEMM (gemm.hip) --------------------------------------------------------
// A row-major fp32 matrix; `trans` reads it transposed (logical (i, j) is
// physical (j, i)).
struct MatView {
  const float* p = nullptr;
  int64_t ld = 0;
  int32_t trans = 0;
  // optional ReLU mask of the same shape and stride: element (i, j) reads as
  // p(i, j) if mask(i, j) > 0, else 0
  const float* mask = nullptr;
  // the operand is stored as bf16 at p16 instead (needs bf16 products, no mask)
  int32_t bf16 = 0;
  const uint16_t* p16 = nullptr;
};
// Output: up to two row-major parts joined along `axis` (0 = rows, 1 =
// columns) at `split`.
struct OutView {
  float* p0 = nullptr;
  float* p1 = nullptr;
  int64_t ld0 = 0, ld1 = 0;
  int32_t split = 1 << 30;
  int32_t axis = 1;
  // optional: the same launch also zeroes rows [*zero_lo (0 if null),
  // min(*zero_hi, zero_cap)) x zero_cols of zero_p (row stride zero_ld; both
  // multiples of 4), a region the GEMM itself does not write
  float* zero_p = nullptr;
  int64_t zero_ld = 0;
  int32_t zero_cols = 0;
  const int32_t* zero_lo = nullptr;
  const int32_t* zero_hi = nullptr;
  int32_t zero_cap = 0;
  // optional: fill ranges done by the same launch (outside the GEMM's output)
  FillPair fills;
  // products on bf16 operands (both factors rounded to nearest even) with
  // fp32 accumulation, on the bf16 MFMA; else fp32 MFMA
  int32_t bf16 = 0;
};
// C[M x N] = A[M x K] B[K x N] with fp32 MFMA (bf16 MFMA with C.bf16).  M (or K when k_dev is set)
// may be read from device memory: m_dev / k_dev point to an int32 count
// (the host values m_cap / k_cap bound the launch).  epilogue: 0 store,
// 1 relu + store, 2 atomic add (C must be zeroed first); with epilogue 2 and
// split_min_chunk > 0 the reduction is split into chunks of at least that
// length over as many blocks as fill the GPU.
// `name` labels the launch for tracing ("gemm_fwd", "gemm_dw", "gemm_dx").
int launch_gemm(const MatView& A, const MatView& B, const OutView& C, int32_t m_cap, int32_t N,
                int32_t k_cap, const int32_t* m_dev, const int32_t* k_dev, int32_t epilogue,
                int32_t split_min_chunk, const char* name, hipStream_t st);
// The arguments of one launch_gemm, for launch_gemm_pair.
struct GemmSpec {
  MatView A, B;
  OutView C;
  int32_t m_cap, N, k_cap;
  const int32_t* m_dev;
  const int32_t* k_dev;
  int32_t epilogue, split_min_chunk;
  const char* name;  // its trace name when launched on its own
};
// Two independent products: one launch (trace name `name`) when they are a
// hidden layer's weight and input gradients (the latency-bound grids then
// share the GPU instead of running one after the other), else launch_gemm
// each.  Neither may write what the other reads.
int launch_gemm_pair(const GemmSpec& p1, const GemmSpec& p2, const char* name, hipStream_t st);

// ---- thin layer-1 products on bf16 operands (gemm_thin.hip) -------------------
// Z = X W (ReLU optional): X [m x K] bf16 (row stride ldx), W [K x N] fp32
// (row stride ldw), Z fp32 (row stride ldo); live rows min(m_cap, *m_dev).
// thin_fwd_ok: the shape and alignment the kernel takes (K % 8 == 0, K <=
// 256, N % 4 == 0, N <= 256, 16-byte rows).  The launch also does `fills`.
// With wt (thin_fwd_wt_elems(K) bf16, 16-byte aligned, written by a WtJob
// earlier on the stream from the same W), every CU copies the staged W^T
// from there instead of converting W itself.
bool thin_fwd_ok(const uint16_t* X, int64_t ldx, const float* W, int64_t ldw, const float* out,
                 int64_t ldo, int32_t K, int32_t N);
int launch_thin_fwd(const uint16_t* X, int64_t ldx, const float* W, int64_t ldw, float* out,
                    int64_t ldo, int32_t m_cap, const int32_t* m_dev, int32_t K, int32_t N, bool relu,
                    const FillPair& fills, const char* name, hipStream_t st,
                    const uint16_t* wt = nullptr);

// The forward's staged W^T: kThinFwdCols rows of thin_fwd_kp(K) bf16 values,
// row n holding W[k][n] for k < K rounded to nearest even, zeros past K and
// in rows n >= N (16-byte rows, the pad keeps the MFMA operand reads free of
// bank conflicts).
constexpr int kThinFwdCols = 256;
__host__ __device__ constexpr int thin_fwd_ks(int32_t K) {
  return K <= 32 ? 2 : K <= 64 ? 4 : K <= 128 ? 8 : K <= 256 ? 16 : 0;
}
__host__ __device__ constexpr int thin_fwd_kp(int32_t K) { return thin_fwd_ks(K) * 16 + 8; }
constexpr int64_t thin_fwd_wt_elems(int32_t K) { return (int64_t)kThinFwdCols * thin_fwd_kp(K); }

// Writes that W^T into wt, for spare blocks of an earlier launch on the same
// stream (the layer-1 aggregation): block `block` of `blocks`.  Threads take
// 8-row chunks of one column, consecutive threads consecutive columns (the
// reads of W are coalesced rows; each thread writes one 16-byte piece).
struct WtJob {
  const float* W = nullptr;
  int64_t ldw = 0;
  int32_t K = 0, N = 0;
  uint16_t* wt = nullptr;
};
__device__ __forceinline__ void run_wt_job(const WtJob& j, int64_t block, int64_t blocks, int threads) {
  const int32_t kp = thin_fwd_kp(j.K), kc = kp / 8;
  const int64_t chunks = (int64_t)kThinFwdCols * kc;
  for (int64_t c = block * threads + threadIdx.x; c < chunks; c += blocks * threads) {
    const int32_t n = (int32_t)(c % kThinFwdCols), k0 = 8 * (int32_t)(c / kThinFwdCols);
    uint16_t v[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int32_t k = k0 + i;
      const float x = (n < j.N && k < j.K) ? j.W[(int64_t)k * j.ldw + n] : 0.f;
      v[i] = __builtin_bit_cast(uint16_t, (__bf16)x);  // nearest even
    }
    uint4 o;
    o.x = (uint32_t)v[0] | ((uint32_t)v[1] << 16);
    o.y = (uint32_t)v[2] | ((uint32_t)v[3] << 16);
    o.z = (uint32_t)v[4] | ((uint32_t)v[5] << 16);
    o.w = (uint32_t)v[6] | ((uint32_t)v[7] << 16);
    *reinterpret_cast<uint4*>(j.wt + (int64_t)n * kp + k0) = o;
  }
}
// spare blocks that do the conversion in reasonable time beside other work
constexpr int kWtJobBlocks = 32;
// dW = X^T Z as nparts partial sums part[c * kw * N + i * N + j] over chunks
// of the live rows: X [m x kw] bf16 (row stride ldx), Z [m x N] bf16 (row
// stride ldz).  thin_dw_parts: the chunk count for m_cap rows (<= 32).
int32_t thin_dw_parts(int32_t m_cap);
bool thin_dw_ok(const uint16_t* X, int64_t ldx, const uint16_t* Z, int64_t ldz, int32_t kw, int32_t N);
int launch_thin_dw(const uint16_t* X, int64_t ldx, const uint16_t* Z, int64_t ldz, int32_t m_cap,
                   const int32_t* m_dev, int32_t kw, int32_t N, float* part, int32_t nparts,
                   const char* name, hipStream_t st);

// ---- output layer + loss (head.hip) ------------------------------------------
// For rows i < B of the last layer's input X [B x K] (K <= 512, a multiple of
// 4; 16-byte aligned): logits Z = X W (W [K x C], 4 <= C <= kHeadMaxClasses; W 16-byte aligned), the
// softmax cross-entropy of row i against labels[label_rows ? label_rows[i] :
// i] (row_loss[i]; dlogits = d(mean loss)/dZ), the tile-wise weight gradient
// dw_part[t] = X_t^T dZ_t over tiles t of kHeadRows rows ([ceil(B / 16) x K x
// C], summed by the SGD launch), and, if dx0 is set, dX = dZ W^T with columns
// < split written to dx0 (row stride ld0) and the rest to dx1 (ld1).  The same
// launch zeroes rows [*zero_lo (0 if null), min(*zero_hi, zero_cap)) x
// zero_cols of zero_p (row stride zero_ld; multiples of 4), if set.
constexpr int kHeadRows = 16;
constexpr int kHeadMinClasses = 4;
constexpr int kHeadMaxClasses = 64;
constexpr int kHeadMaxParts = 4;  // input width cut into parts of 128 (512 / 128)
struct HeadJob {
  const float* X = nullptr;
  int32_t K = 0;
  const float* W = nullptr;
  int32_t C = 0;
  const int32_t* labels = nullptr;
  int64_t n_labels = 0;
  const int32_t* label_rows = nullptr;
  int32_t B = 0;
  float* logits = nullptr;
  float* dlogits = nullptr;
  float* row_loss = nullptr;
  float* dw_part = nullptr;
  float* dx0 = nullptr;
  float* dx1 = nullptr;
  int32_t split = 1 << 30;
  int32_t ld0 = 0, ld1 = 0;
  float* zero_p = nullptr;
  int32_t zero_ld = 0, zero_cols = 0;
  const int32_t* zero_lo = nullptr;
  const int32_t* zero_hi = nullptr;
  int32_t zero_cap = 0;
  // optional exchange buffers of the split form (head_xch_elems floats,
  // head_sync_words int32 that must be zero before the first launch and are
  // left zero by every launch); without them one block takes a whole row tile
  float* xch = nullptr;
  int32_t* sync = nullptr;
};
int launch_head(const HeadJob& j, hipStream_t st);
int64_t head_part_elems(int32_t B, int32_t K, int32_t C);
int64_t head_xch_elems(int32_t B);
int64_t head_sync_words(int32_t B);

// ---- loss / sgd (loss.hip) -----------------------------------------------------
// Gradient of parameters [off, off + len) given as nb partial sums
// p[b * len + i]; the SGD launch adds them in a fixed order and also stores
// the sum into g.  Up to two such ranges (they must not overlap).
struct GradRange {
  const float* p = nullptr;
  int64_t off = 0, len = 0;
  int32_t nb = 0;
};
struct GradParts {
  GradRange r[2];
};
// label_i = labels[rows ? rows[i] : i]; rows[i] must lie in [0, n_labels).
int launch_softmax_xent(const float* logits, const int32_t* labels, int64_t n_labels,
                        const int32_t* rows, int32_t B, int32_t C, int32_t ld, float* dlogits,
                        float* row_loss, hipStream_t st);
// Adam's state, its factors (a1 = 1 - b1, a2 = 1 - b2, rounded from double)
// and this step's bias corrections c1 = 1 / (1 - beta1^t), c2 = 1 / (1 -
// beta2^t); m == nullptr means plain SGD.
struct AdamJob {
  float* m = nullptr;
  float* v = nullptr;
  float b1 = 0.f, a1 = 0.f, b2 = 0.f, a2 = 0.f, eps = 0.f, c1 = 1.f, c2 = 1.f;
};
int launch_sgd(float* w, float* g, int64_t n, float lr, const float* row_loss, int32_t B,
               float* loss_out, hipStream_t st, const GradParts& parts = GradParts{},
               const AdamJob& adam = AdamJob{});

}  // namespace gnn
