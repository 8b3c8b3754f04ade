// Loss and optimiser of the training step (paper section 2.2, eq. (3)): the
// mean over the batch of the per-root softmax cross-entropy, its gradient
// w.r.t. the logits, and a plain SGD update of every parameter.
#include <mutex>

#include "internal.hpp"
#include "wave.hpp"

namespace gnn {

namespace {

constexpr int kThreads = 256;
constexpr int kMaxC = 256;  // classes per row handled by one wave (4 per lane)

// One wave per row: label_i = labels[rows ? rows[i] : i].
__global__ void __launch_bounds__(kThreads)
softmax_xent_kernel(const float* __restrict__ logits, const int32_t* __restrict__ labels,
                    int64_t n_labels, const int32_t* __restrict__ rows, int32_t B, int32_t C,
                    int32_t ld,
                    float* __restrict__ dlogits, float* __restrict__ row_loss, int* err) {
  const int lane = lane_id();
  const int64_t i = ((int64_t)blockIdx.x * kThreads + threadIdx.x) >> 6;
  if (i >= B) return;
  const int64_t li = rows ? rows[i] : i;
  const int32_t y = (li >= 0 && li < n_labels) ? labels[li] : -1;
  const float* z = logits + i * (int64_t)ld;
  float v[kMaxC / 64];
  float mx = -INFINITY;
#pragma unroll
  for (int t = 0; t < kMaxC / 64; ++t) {
    const int c = lane + 64 * t;
    v[t] = c < C ? z[c] : -INFINITY;
    mx = fmaxf(mx, v[t]);
  }
  mx = wave_max(mx);
  float s = 0.f;
#pragma unroll
  for (int t = 0; t < kMaxC / 64; ++t) {
    const int c = lane + 64 * t;
    v[t] = c < C ? expf(v[t] - mx) : 0.f;
    s += v[t];
  }
  s = wave_sum(s);
  const bool ok = y >= 0 && y < C;
  if (!ok && lane == 0) set_device_error(err, GNN_DEVERR_LABEL_RANGE);
  const float inv_s = 1.f / s, inv_b = 1.f / (float)B;
  float* d = dlogits + i * (int64_t)ld;
#pragma unroll
  for (int t = 0; t < kMaxC / 64; ++t) {
    const int c = lane + 64 * t;
    if (c < C) d[c] = ok ? (v[t] * inv_s - (c == y ? 1.f : 0.f)) * inv_b : 0.f;
  }
  if (lane == 0) row_loss[i] = ok ? (logf(s) + mx - z[y]) : 0.f;
}

// The update of parameter i with gradient g: SGD, or Adam with its moments.
__device__ __forceinline__ void update(float* __restrict__ w, int64_t i, float g, float lr,
                                       const AdamJob& a) {
  if (!a.m) {
    w[i] -= lr * g;
    return;
  }
  const float m = a.b1 * a.m[i] + a.a1 * g;
  const float v = a.b2 * a.v[i] + a.a2 * g * g;
  a.m[i] = m;
  a.v[i] = v;
  w[i] -= lr * (m * a.c1) / (sqrtf(v * a.c2) + a.eps);
}

// w -= lr * g (or Adam).  Over each range of `parts`, g is first summed from
// its partials (and stored) by the blocks past upd_blocks (those of range 0,
// then those of range 1): 64 parameters per block, each summed by 4 waves
// over every 4th partial and the 4 sums added in wave order (a fixed order).
// Block 0 also sums row_loss in a fixed order into *loss_out.
constexpr int kPartCols = 64;
__global__ void __launch_bounds__(kThreads)
sgd_kernel(float* __restrict__ w, float* __restrict__ g, int64_t n, float lr,
           const float* __restrict__ row_loss, int32_t B, float* __restrict__ loss_out,
           GradParts gp, int32_t upd_blocks, int32_t blocks0, AdamJob adam) {
  if ((int32_t)blockIdx.x >= upd_blocks) {
    __shared__ float red[kThreads / 64][kPartCols];
    const int32_t pb = (int32_t)blockIdx.x - upd_blocks;
    const bool second = pb >= blocks0;
    const GradRange parts = second ? gp.r[1] : gp.r[0];
    const int c = threadIdx.x & 63, grp = threadIdx.x >> 6;
    const int64_t pi = (int64_t)(second ? pb - blocks0 : pb) * kPartCols + c;
    float acc = 0.f;
    if (pi < parts.len) {
      const float* p = parts.p + pi;
      int32_t b = grp;
      for (; b + 12 < parts.nb; b += 16) {
        const float v0 = p[(int64_t)b * parts.len], v1 = p[(int64_t)(b + 4) * parts.len];
        const float v2 = p[(int64_t)(b + 8) * parts.len], v3 = p[(int64_t)(b + 12) * parts.len];
        acc += v0;
        acc += v1;
        acc += v2;
        acc += v3;
      }
      for (; b < parts.nb; b += 4) acc += p[(int64_t)b * parts.len];
    }
    red[grp][c] = acc;
    __syncthreads();
    if (grp == 0 && pi < parts.len) {
      float t = 0.f;
#pragma unroll
      for (int k = 0; k < kThreads / 64; ++k) t += red[k][c];
      const int64_t i = parts.off + pi;
      g[i] = t;
      update(w, i, t, lr, adam);
    }
    return;
  }
  for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < n;
       i += (int64_t)upd_blocks * kThreads) {
    const int64_t p0 = i - gp.r[0].off, p1 = i - gp.r[1].off;
    if ((p0 < 0 || p0 >= gp.r[0].len) && (p1 < 0 || p1 >= gp.r[1].len)) update(w, i, g[i], lr, adam);
  }
  if (blockIdx.x != 0 || !loss_out) return;
  __shared__ float part[kThreads / 64];
  float s = 0.f;
  for (int32_t i = threadIdx.x; i < B; i += kThreads) s += row_loss[i];
  s = wave_sum(s);
  if (lane_id() == 0) part[threadIdx.x >> 6] = s;
  __syncthreads();
  if (threadIdx.x == 0) {
    float t = 0.f;
    for (int k = 0; k < kThreads / 64; ++k) t += part[k];
    *loss_out = B > 0 ? t / (float)B : 0.f;
  }
}

}  // namespace

int launch_softmax_xent(const float* logits, const int32_t* labels, int64_t n_labels,
                        const int32_t* rows, int32_t B, int32_t C, int32_t ld, float* dlogits,
                        float* row_loss, hipStream_t st) {
  if (B <= 0) return GNN_OK;
  if (C > kMaxC) return fail(GNN_EINVAL, "softmax: %d classes > %d", C, kMaxC);
  const unsigned grid = (unsigned)ceil_div((int64_t)B * 64, kThreads);
  launch("softmax_xent", softmax_xent_kernel, grid, kThreads, 0, st, logits, labels, n_labels, rows,
         B, C, ld, dlogits, row_loss, device_error_word());
  GNN_LAUNCH_CHECK("softmax cross-entropy");
  return GNN_OK;
}

int launch_sgd(float* w, float* g, int64_t n, float lr, const float* row_loss, int32_t B,
               float* loss_out, hipStream_t st, const GradParts& parts, const AdamJob& adam) {
  for (const GradRange& r : parts.r)
    if (r.len && (r.off < 0 || r.off + r.len > n || r.nb < 1 || !r.p))
      return fail(GNN_EINVAL, "sgd: bad gradient partials");
  const GradRange &r0 = parts.r[0], &r1 = parts.r[1];
  if (r0.len && r1.len && r0.off < r1.off + r1.len && r1.off < r0.off + r0.len)
    return fail(GNN_EINVAL, "sgd: overlapping gradient partials");
  int64_t blocks = ceil_div(n, kThreads * 4);
  blocks = blocks < 1 ? 1 : (blocks > 1024 ? 1024 : blocks);
  const int64_t pb0 = r0.len ? ceil_div(r0.len, kPartCols) : 0;
  const int64_t pb1 = r1.len ? ceil_div(r1.len, kPartCols) : 0;
  launch("sgd", sgd_kernel, (unsigned)(blocks + pb0 + pb1), kThreads, 0, st, w, g, n, lr, row_loss, B,
         loss_out, parts, (int32_t)blocks, (int32_t)pb0, adam);
  GNN_LAUNCH_CHECK("sgd");
  return GNN_OK;
}

// Scratch of gnn_softmax_xent_noalloc: the per-row losses of one call, in a
// library-owned array (one per GPU, held until the process ends).  Host code
// uses the address hipGetSymbolAddress returns for the current device, never
// the array's name.
__device__ __align__(256) float scratch[GNN_XENT_NOALLOC_MAX_ROWS];

// Device address of `scratch` on the current device (looked up once per
// device, with that device current), or null.
float* scratch_ptr() {
  static std::mutex mu;
  static float* addr[64] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return nullptr;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess) return nullptr;
    addr[dev] = static_cast<float*>(p);
  }
  return addr[dev];
}

}  // namespace gnn

extern "C" {

size_t gnn_loss_workspace_bytes(int32_t B) { return (size_t)(B > 0 ? B : 1) * sizeof(float) + 256; }

int gnn_softmax_xent(const float* logits, const int32_t* labels, int32_t B, int32_t C,
                     float* dlogits, float* loss_out, void* ws, size_t ws_bytes, void* stream) {
  using namespace gnn;
  if (!logits || !labels || !dlogits || !loss_out || !ws)
    return fail(GNN_EINVAL, "gnn_softmax_xent: null pointer");
  if (B < 0 || C < 1 || C > kMaxC) return fail(GNN_EINVAL, "gnn_softmax_xent: bad B or C");
  if (ws_bytes < gnn_loss_workspace_bytes(B)) return fail(GNN_EWORKSPACE, "gnn_softmax_xent: workspace");
  hipStream_t st = as_stream(stream);
  float* row_loss = static_cast<float*>(ws);
  if (int rc = launch_softmax_xent(logits, labels, B, nullptr, B, C, C, dlogits, row_loss, st))
    return rc;
  return launch_sgd(nullptr, nullptr, 0, 0.f, row_loss, B, loss_out, st);
}

int gnn_softmax_xent_noalloc(const float* logits, const int32_t* labels, int32_t B, int32_t C,
                             float* dlogits, float* loss_out, void* stream) {
  using namespace gnn;
  if (!logits || !labels || !dlogits || !loss_out)
    return fail(GNN_EINVAL, "gnn_softmax_xent_noalloc: null pointer");
  if (B < 0 || C < 1 || C > kMaxC) return fail(GNN_EINVAL, "gnn_softmax_xent_noalloc: bad B or C");
  if (B > GNN_XENT_NOALLOC_MAX_ROWS)
    return fail(GNN_EINVAL, "gnn_softmax_xent_noalloc: %d rows > %d (the library's scratch)", B,
                GNN_XENT_NOALLOC_MAX_ROWS);
  float* row_loss = scratch_ptr();
  if (!row_loss) return fail(GNN_EHIP, "gnn_softmax_xent_noalloc: scratch address unavailable");
  hipStream_t st = as_stream(stream);
  // every row's loss is written before the mean reads it: nothing to clear
  if (int rc = launch_softmax_xent(logits, labels, B, nullptr, B, C, C, dlogits, row_loss, st))
    return rc;
  return launch_sgd(nullptr, nullptr, 0, 0.f, row_loss, B, loss_out, st);
}

int gnn_sgd(float* w, const float* g, int64_t n, float lr, void* stream) {
  using namespace gnn;
  if (n < 0 || (n > 0 && (!w || !g))) return fail(GNN_EINVAL, "gnn_sgd: bad arguments");
  if (n == 0) return GNN_OK;
  // without partials the kernel only reads g
  return launch_sgd(w, const_cast<float*>(g), n, lr, nullptr, 0, nullptr, as_stream(stream));
}

}  // extern "C"
