// Feature fetch: out[i, :] = X[ids[i], :] (the "data fetching" step of a
// mini-batch, paper section 2.2).  Every thread moves 16-byte chunks
// (global_load_dwordx4 / global_store_dwordx4); consecutive threads cover
// consecutive chunks of a row and consecutive rows, so the stores are fully
// coalesced and each source row is read as one contiguous burst.
#include "internal.hpp"
#include "wave.hpp"

namespace gnn {

namespace {

constexpr int kThreads = 256;
constexpr int kUnroll = 4;

// Blocks past gather_blocks run the sampling call's last step (if any).
__global__ void __launch_bounds__(kThreads)
gather_kernel(const uint4* __restrict__ X, int64_t n_rows, int64_t ld_x16,
              const int32_t* __restrict__ ids,
              const int32_t* n_ids, int32_t cap, int32_t cpr, uint4* __restrict__ out,
              int64_t ld_out16, int* err, int32_t gather_blocks, SampleTail tail) {
  if ((int32_t)blockIdx.x >= gather_blocks) {
    finish_sampling(tail, blockIdx.x - gather_blocks, gridDim.x - gather_blocks, kThreads);
    return;
  }
  int32_t n = *n_ids;
  if (n > cap) {
    if (blockIdx.x == 0 && threadIdx.x == 0) set_device_error(err, GNN_DEVERR_CAPACITY);
    n = cap;
  }
  // chunk counts fit 32 bits (checked on the host)
  const uint32_t total = (uint32_t)n * (uint32_t)cpr;
  const uint32_t ucpr = (uint32_t)cpr;
  const uint32_t stride = (uint32_t)gather_blocks * kThreads;
  uint32_t c = blockIdx.x * kThreads + threadIdx.x;
  for (; c + (kUnroll - 1) * stride < total; c += kUnroll * stride) {
    uint4 v[kUnroll];
    uint32_t r[kUnroll], j[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const uint32_t cc = c + u * stride;
      r[u] = cc / ucpr;
      j[u] = cc - r[u] * ucpr;
      const int32_t id = ids[r[u]];
      if (id >= 0 && id < n_rows) {
        v[u] = X[(int64_t)id * ld_x16 + j[u]];
      } else {
        v[u] = make_uint4(0, 0, 0, 0);
        set_device_error(err, GNN_DEVERR_SEED_RANGE);
      }
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) out[(int64_t)r[u] * ld_out16 + j[u]] = v[u];
  }
  for (; c < total; c += stride) {
    const uint32_t r = c / ucpr, j = c - r * ucpr;
    const int32_t id = ids[r];
    uint4 v = make_uint4(0, 0, 0, 0);
    if (id >= 0 && id < n_rows) v = X[(int64_t)id * ld_x16 + j];
    else set_device_error(err, GNN_DEVERR_SEED_RANGE);
    out[(int64_t)r * ld_out16 + j] = v;
  }
}

}  // namespace

int launch_gather(const void* X, int32_t esize, int64_t n_rows, int64_t ld_x, int32_t F,
                  const int32_t* ids, const int32_t* n_ids, int32_t cap, void* out, int64_t ld_out,
                  const SampleTail* tail, hipStream_t st) {
  const int64_t row_bytes = (int64_t)F * esize;
  const int32_t cpr = (int32_t)(row_bytes / 16);
  const int64_t chunks = (int64_t)cap * cpr;
  int64_t blocks = ceil_div(chunks, (int64_t)kThreads * kUnroll);
  blocks = blocks < 1 ? 1 : (blocks > 8192 ? 8192 : blocks);
  int64_t tblocks = 0;
  SampleTail t{};
  if (tail) {
    t = *tail;
    tblocks = 512;
  }
  launch("gather", gather_kernel, (unsigned)(blocks + tblocks), kThreads, 0, st,
         static_cast<const uint4*>(X), n_rows, ld_x * esize / 16, ids, n_ids, cap, cpr,
         static_cast<uint4*>(out), ld_out * esize / 16, device_error_word(), (int32_t)blocks, t);
  GNN_LAUNCH_CHECK("gather");
  return GNN_OK;
}

}  // namespace gnn

extern "C" int gnn_gather_features(const void* X, int32_t dtype, int64_t n_rows, int64_t ld_x,
                                   int32_t F, const int32_t* ids, const int32_t* n_ids, int32_t cap,
                                   void* out, int64_t ld_out, void* stream) {
  using namespace gnn;
  if (!X || !ids || !n_ids || !out) return fail(GNN_EINVAL, "gnn_gather_features: null pointer");
  if (dtype != GNN_F32 && dtype != GNN_BF16) return fail(GNN_EINVAL, "gnn_gather_features: bad dtype");
  if (F <= 0 || cap < 0 || n_rows < 0) return fail(GNN_EINVAL, "gnn_gather_features: bad size");
  const int32_t es = dtype == GNN_F32 ? 4 : 2;
  if (((int64_t)F * es) % 16 || (ld_x * es) % 16 || (ld_out * es) % 16 || ld_x < F || ld_out < F)
    return fail(GNN_EINVAL, "gnn_gather_features: rows and strides must be 16-byte multiples");
  if ((reinterpret_cast<uintptr_t>(X) | reinterpret_cast<uintptr_t>(out)) & 15)
    return fail(GNN_EINVAL, "gnn_gather_features: pointers must be 16-byte aligned");
  if ((int64_t)cap * ((int64_t)F * es / 16) + 8LL * 8192 * 256 >= (1LL << 32))
    return fail(GNN_EINVAL, "gnn_gather_features: cap * row chunks too large");
  if (cap == 0) return GNN_OK;
  return launch_gather(X, es, n_rows, ld_x, F, ids, n_ids, cap, out, ld_out, nullptr,
                       as_stream(stream));
}
