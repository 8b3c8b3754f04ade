// Error reporting, the sticky device error word, device-wide scan and fill.
#include <cstdarg>
#include <cstdio>
#include <mutex>

#include "internal.hpp"
#include "wave.hpp"

namespace gnn {

static thread_local char g_msg[512] = "";

int fail(int code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_msg, sizeof g_msg, fmt, ap);
  va_end(ap);
  return code;
}

int hip_fail(hipError_t e, const char* what) {
  return fail(GNN_EHIP, "%s: %s", what, hipGetErrorString(e));
}

// One word per device; bits are GNN_DEVERR_*.
__device__ int g_device_error[1];

int* device_error_word() {
  static std::mutex mu;
  static int* addr[64] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return nullptr;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(g_device_error)) != hipSuccess) return nullptr;
    addr[dev] = static_cast<int*>(p);
  }
  return addr[dev];
}

// ---------------------------------------------------------------------------
// Device-wide exclusive scan: reduce tiles, scan tile sums, scan tiles.
// ---------------------------------------------------------------------------
constexpr int SCAN_THREADS = 256;
constexpr int SCAN_ITEMS = 8;
constexpr int SCAN_TILE = SCAN_THREADS * SCAN_ITEMS;

size_t scan_scratch_ints(int64_t cap) { return (size_t)ceil_div(cap, SCAN_TILE) + 1; }

__device__ inline int64_t clamp_n(const int32_t* n_dev, int64_t cap) {
  int64_t n = *n_dev;
  return n < 0 ? 0 : (n > cap ? cap : n);
}

// Block-wide exclusive scan of one value per thread; returns the block total in *total.
__device__ inline int32_t block_exclusive_scan(int32_t x, int32_t* total) {
  __shared__ int32_t wsum[SCAN_THREADS / 64];
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  int32_t inc = wave_inclusive_scan(x);
  if (lane == 63) wsum[wid] = inc;
  __syncthreads();
  int32_t off = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < SCAN_THREADS / 64; ++w) {
    off += (w < wid) ? wsum[w] : 0;
    tot += wsum[w];
  }
  __syncthreads();
  *total = tot;
  return off + inc - x;
}

__global__ void __launch_bounds__(SCAN_THREADS)
scan_reduce_kernel(const int32_t* __restrict__ in, const int32_t* n_dev, int64_t cap,
                   int32_t* __restrict__ partial) {
  const int64_t n = clamp_n(n_dev, cap);
  const int64_t base = (int64_t)blockIdx.x * SCAN_TILE;
  if (base >= n && blockIdx.x != 0) return;
  int32_t s = 0;
#pragma unroll
  for (int i = 0; i < SCAN_ITEMS; ++i) {
    int64_t idx = base + (int64_t)i * SCAN_THREADS + threadIdx.x;
    if (idx < n) s += in[idx];
  }
  int32_t tot;
  block_exclusive_scan(s, &tot);
  if (threadIdx.x == 0) partial[blockIdx.x] = tot;
}

__global__ void __launch_bounds__(1024)
scan_partials_kernel(int32_t* partial, const int32_t* n_dev, int64_t cap, int32_t* out,
                     int32_t* total_dst) {
  const int64_t n = clamp_n(n_dev, cap);
  const int64_t nb = (n + SCAN_TILE - 1) / SCAN_TILE;
  __shared__ int32_t wsum[16];
  __shared__ int32_t carry_s;
  if (threadIdx.x == 0) carry_s = 0;
  __syncthreads();
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  for (int64_t c = 0; c < nb; c += 1024) {
    int64_t i = c + threadIdx.x;
    int32_t x = (i < nb) ? partial[i] : 0;
    int32_t inc = wave_inclusive_scan(x);
    if (lane == 63) wsum[wid] = inc;
    __syncthreads();
    int32_t off = carry_s, tot = 0;
    for (int w = 0; w < 16; ++w) {
      off += (w < wid) ? wsum[w] : 0;
      tot += wsum[w];
    }
    if (i < nb) partial[i] = off + inc - x;
    __syncthreads();
    if (threadIdx.x == 0) carry_s += tot;
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    out[n] = carry_s;
    if (total_dst) *total_dst = carry_s;
  }
}

__global__ void __launch_bounds__(SCAN_THREADS)
scan_apply_kernel(const int32_t* __restrict__ in, const int32_t* n_dev, int64_t cap,
                  const int32_t* __restrict__ partial, int32_t* __restrict__ out) {
  const int64_t n = clamp_n(n_dev, cap);
  const int64_t base = (int64_t)blockIdx.x * SCAN_TILE;
  if (base >= n) return;
  // each thread owns SCAN_ITEMS consecutive items
  const int64_t first = base + (int64_t)threadIdx.x * SCAN_ITEMS;
  int32_t v[SCAN_ITEMS];
  int32_t s = 0;
#pragma unroll
  for (int i = 0; i < SCAN_ITEMS; ++i) {
    v[i] = (first + i < n) ? in[first + i] : 0;
    s += v[i];
  }
  int32_t tot;
  int32_t off = block_exclusive_scan(s, &tot) + partial[blockIdx.x];
#pragma unroll
  for (int i = 0; i < SCAN_ITEMS; ++i) {
    if (first + i < n) out[first + i] = off;
    off += v[i];
  }
}

int launch_exclusive_scan(const int32_t* in, int32_t* out, const int32_t* n_dev, int64_t cap,
                          int32_t* total_dst, int32_t* scratch, hipStream_t st) {
  const int64_t nb = ceil_div(cap > 0 ? cap : 1, SCAN_TILE);
  scan_reduce_kernel<<<dim3((unsigned)nb), SCAN_THREADS, 0, st>>>(in, n_dev, cap, scratch);
  scan_partials_kernel<<<1, 1024, 0, st>>>(scratch, n_dev, cap, out, total_dst);
  scan_apply_kernel<<<dim3((unsigned)nb), SCAN_THREADS, 0, st>>>(in, n_dev, cap, scratch, out);
  GNN_LAUNCH_CHECK("exclusive scan");
  return GNN_OK;
}

// ---------------------------------------------------------------------------
// Fill: up to 8 ranges of 32-bit words in one launch (used instead of
// hipMemsetAsync so that a captured graph replays correctly).
// ---------------------------------------------------------------------------
struct FillArgs {
  int32_t* p[8];
  int64_t n[8];
  int32_t v[8];
};

__global__ void __launch_bounds__(256) fill_kernel(FillArgs a) {
  const int r = blockIdx.y;
  int32_t* p = a.p[r];
  const int64_t n = a.n[r];
  const int32_t v = a.v[r];
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256)
    p[i] = v;
}

int launch_fill(const FillRange* ranges, int n, hipStream_t st) {
  if (n <= 0) return GNN_OK;
  if (n > 8) return fail(GNN_EINVAL, "launch_fill: too many ranges");
  FillArgs a{};
  int64_t mx = 0;
  for (int i = 0; i < n; ++i) {
    a.p[i] = static_cast<int32_t*>(ranges[i].p);
    a.n[i] = ranges[i].p ? ranges[i].n_words : 0;
    a.v[i] = ranges[i].value;
    mx = a.n[i] > mx ? a.n[i] : mx;
  }
  if (mx == 0) return GNN_OK;
  int64_t blocks = ceil_div(mx, 256 * 4);
  blocks = blocks > 2048 ? 2048 : (blocks < 1 ? 1 : blocks);
  fill_kernel<<<dim3((unsigned)blocks, (unsigned)n), 256, 0, st>>>(a);
  GNN_LAUNCH_CHECK("fill");
  return GNN_OK;
}

}  // namespace gnn

extern "C" {

const char* gnn_last_error(void) { return gnn::g_msg; }

const char* gnn_version(void) { return "gnnhip 0.1 (gfx950)"; }

int gnn_check_errors(void* stream, int32_t* bits) {
  using namespace gnn;
  if (bits) *bits = 0;
  hipStream_t st = as_stream(stream);
  GNN_HIP_TRY(hipStreamSynchronize(st));
  int* w = device_error_word();
  if (!w) return fail(GNN_EHIP, "device error word unavailable");
  int host = 0;
  GNN_HIP_TRY(hipMemcpy(&host, w, sizeof(int), hipMemcpyDeviceToHost));
  if (host != 0) {
    int zero = 0;
    GNN_HIP_TRY(hipMemcpy(w, &zero, sizeof(int), hipMemcpyHostToDevice));
    if (bits) *bits = host;
    return fail(GNN_EDEVICE, "device-side error bits 0x%x", host);
  }
  return GNN_OK;
}

}  // extern "C"
