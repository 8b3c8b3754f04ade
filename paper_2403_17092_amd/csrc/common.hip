// Error reporting, the sticky device error word, launch tracing and fill.
#include <cstdarg>
#include <cstdio>
#include <cstring>
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

// ---------------------------------------------------------------------------
// Launch tracing: the installed trace of the calling thread, if any.
// ---------------------------------------------------------------------------
static thread_local gnn_trace* g_trace = nullptr;

bool trace_slot(const char* name, hipEvent_t* start, hipEvent_t* stop) {
  gnn_trace* t = g_trace;
  if (!t || (t->only && std::strcmp(t->only, name) != 0)) return false;
  const int i = t->count;
  if (i >= t->capacity || !t->events || !t->events[2 * i] || !t->events[2 * i + 1]) {
    ++t->dropped;
    return false;
  }
  *start = static_cast<hipEvent_t>(t->events[2 * i]);
  *stop = static_cast<hipEvent_t>(t->events[2 * i + 1]);
  if (t->names) t->names[i] = name;
  ++t->count;
  return true;
}

int device_cu_count() {
  static std::mutex mu;
  static int count[64] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  std::lock_guard<std::mutex> lock(mu);
  if (!count[dev]) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n < 1)
      n = 256;
    count[dev] = n;
  }
  return count[dev];
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
  launch("fill", fill_kernel, dim3((unsigned)blocks, (unsigned)n), 256, 0, st, a);
  GNN_LAUNCH_CHECK("fill");
  return GNN_OK;
}

}  // namespace gnn

extern "C" {

const char* gnn_last_error(void) { return gnn::g_msg; }

const char* gnn_version(void) { return "gnnhip 0.1 (gfx950)"; }

int gnn_trace_begin(gnn_trace* t) {
  if (t && (t->capacity < 0 || (t->capacity > 0 && !t->events)))
    return gnn::fail(GNN_EINVAL, "gnn_trace_begin: bad capacity or events");
  gnn::g_trace = t;
  return GNN_OK;
}

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
