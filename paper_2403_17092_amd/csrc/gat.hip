// GAT layer kernels: one attention head as defined by Velickovic et al.
// (ICLR 2018, eqs. 1-4), one of the message-passing models paper section 2.1
// names.  On a sampled block, dst node v attends over its sampled edges and
// its self edge:
//   T = H W;  pre_vu = a_l . T_v + a_r . T_u;  e_vu = LeakyReLU(pre_vu, 0.2);
//   alpha_vu = exp(e_vu - m_v) / sum_w exp(e_vw - m_v);  out_v = sum_u alpha_vu T_u.
// T comes from a GEMM; these kernels compute the scores s_l = T a_l and
// s_r = T a_r (per src row), the attention sum (one wavefront per dst row,
// keeping m_v and the normaliser's inverse for the backward pass), and the
// backward pass through the softmax:
//   dT_u += alpha_vu dOut_v;  dalpha_vu = dOut_v . T_u;
//   dpre_vu = alpha_vu (dalpha_vu - S_v) lk_vu,  S_v = sum_u alpha_vu dalpha_vu,
//   lk = 1 or 0.2 (LeakyReLU's slope at pre);
//   ds_l[v] = sum_u dpre_vu;  ds_r[u] = sum_v dpre_vu;
//   dT_v += ds_l[v] a_l (dst rows);  dT_u += ds_r[u] a_r.
// The edge pass splits dpre into alpha lk dalpha (known per edge at once) and
// -S_v alpha lk (a second, scalar sweep once S_v is summed), so no per-edge
// intermediate is stored.  Rows of T have a stride padded to 16 bytes; the
// columns past F are never read as values (masked to 0 on load).
#include "internal.hpp"
#include "wave.hpp"

namespace gnn {

namespace {

constexpr int kThreads = 256;
constexpr float kSlope = 0.2f;

__device__ __forceinline__ float leaky(float x) { return x > 0.f ? x : kSlope * x; }

__device__ __forceinline__ bool aligned16(const void* p) {
  return (reinterpret_cast<uintptr_t>(p) & 15) == 0;
}

// Columns 4q .. 4q + 3 of row r (stride ld floats); columns >= F read as 0.
__device__ __forceinline__ float4 load_cols(const float* p, int64_t ld, int64_t r, int q, int32_t F) {
  const int32_t c = 4 * q;
  const float* s = p + r * ld + c;
  if (c + 4 <= F && aligned16(s)) return *reinterpret_cast<const float4*>(s);
  float v[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) v[i] = c + i < F ? s[i] : 0.f;
  return make_float4(v[0], v[1], v[2], v[3]);
}

__device__ __forceinline__ void store_cols(float* p, int64_t ld, int64_t r, int q, int32_t F, float4 x) {
  const int32_t c = 4 * q;
  float* d = p + r * ld + c;
  if (c + 4 <= F && aligned16(d)) {
    *reinterpret_cast<float4*>(d) = x;
    return;
  }
  const float v[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
  for (int i = 0; i < 4; ++i)
    if (c + i < F) d[i] = v[i];
}

__device__ __forceinline__ float dot4(float4 a, float4 b) {
  return a.x * b.x + a.y * b.y + a.z * b.z + a.w * b.w;
}

// Layer 1's input rows: row u of the output = feature row rows[u] (or row u
// with no id list), widened to fp32; ids outside [0, n_rows) give zero rows.
template <int DT>
__global__ void __launch_bounds__(kThreads)
gather_kernel(const void* __restrict__ X, const int32_t* __restrict__ rows, int64_t n_rows, int64_t ld_x,
              const int32_t* counts, int32_t cap, int32_t c4, float4* __restrict__ out) {
  int32_t n = counts[1];
  n = n > cap ? cap : n;
  const int64_t total = (int64_t)n * c4;
  for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * kThreads) {
    const int64_t u = i / c4;
    const int32_t q = (int32_t)(i - u * c4);
    int64_t r = rows ? (int64_t)rows[u] : u;
    float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
    if (r >= 0 && r < n_rows) {
      if (DT == GNN_F32) {
        v = reinterpret_cast<const float4*>(static_cast<const float*>(X) + r * ld_x)[q];
      } else {
        const uint2 w = reinterpret_cast<const uint2*>(static_cast<const uint16_t*>(X) + r * ld_x)[q];
        v = make_float4(__uint_as_float(w.x << 16), __uint_as_float(w.x & 0xFFFF0000u),
                        __uint_as_float(w.y << 16), __uint_as_float(w.y & 0xFFFF0000u));
      }
    }
    out[i] = v;
  }
}

// s[2u] = a_l . T_u, s[2u + 1] = a_r . T_u for every src row u: LG lanes per
// row (64 / LG rows per wave), each lane over every LG-th 4-column chunk.
template <int LG>
__global__ void __launch_bounds__(kThreads)
scores_kernel(const float* __restrict__ T, int32_t ldt, const float* __restrict__ a, int32_t F,
              const int32_t* counts, float* __restrict__ s) {
  const int lane = lane_id();
  const int q0 = lane % LG;
  const int64_t u = (((int64_t)blockIdx.x * kThreads + threadIdx.x) >> 6) * (64 / LG) + lane / LG;
  const bool live = u < counts[1];
  float sl = 0.f, sr = 0.f;
  if (live)
    for (int q = q0; 4 * q < F; q += LG) {
      const float4 t = load_cols(T, ldt, u, q, F);
      sl += dot4(t, load_cols(a, 0, 0, q, F));
      sr += dot4(t, load_cols(a + F, 0, 0, q, F));
    }
#pragma unroll
  for (int d = 1; d < LG; d <<= 1) {
    sl += __shfl_xor(sl, d, 64);
    sr += __shfl_xor(sr, d, 64);
  }
  if (live && q0 == 0) {
    s[2 * u] = sl;
    s[2 * u + 1] = sr;
  }
}

struct EdgeView {
  const int32_t* indptr;
  const int32_t* indices;
  const int32_t* counts;
};

// out_v = sum over v's edges and its self edge of alpha_vu T_u (ReLU if
// `relu`); stats[2v] = m_v, stats[2v + 1] = 1 / sum_u exp(e_vu - m_v).
// LG lanes hold one row (LG = chunks of 4 columns, rounded up to a power of
// two); the wave works on 64 / LG edges at a time.
template <int LG>
__global__ void __launch_bounds__(kThreads)
attend_kernel(EdgeView b, const float* __restrict__ T, int32_t ldt, const float* __restrict__ s,
              int32_t F, int32_t relu, float* __restrict__ out, float* __restrict__ stats) {
  constexpr int G = 64 / LG;
  const int lane = lane_id();
  const int g = lane / LG, q = lane % LG;
  const int64_t v = ((int64_t)blockIdx.x * kThreads + threadIdx.x) >> 6;
  if (v >= b.counts[0]) return;
  const int32_t e0 = b.indptr[v], c = b.indptr[v + 1] - e0;
  const float sl = s[2 * v];
  const float e_self = leaky(sl + s[2 * v + 1]);
  float mx = e_self;
  for (int32_t l = lane; l < c; l += 64) mx = fmaxf(mx, leaky(sl + s[2 * b.indices[e0 + l] + 1]));
  mx = wave_max(mx);
  float den = 0.f;
  for (int32_t l = lane; l < c; l += 64) den += __expf(leaky(sl + s[2 * b.indices[e0 + l] + 1]) - mx);
  den = wave_sum(den) + __expf(e_self - mx);
  const float inv = 1.f / den;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int32_t base = 0; base < c; base += 64) {
    const int32_t cc = c - base < 64 ? c - base : 64;
    int32_t my_u = 0;
    float my_w = 0.f;
    if (lane < cc) {
      my_u = b.indices[e0 + base + lane];
      my_w = __expf(leaky(sl + s[2 * my_u + 1]) - mx) * inv;
    }
    for (int32_t k = 0; k < cc; k += G) {
      const int32_t l = k + g;
      const int32_t u = __shfl(my_u, l & 63, 64);
      const float w = __shfl(my_w, l & 63, 64);
      if (l < cc && 4 * q < F) {
        const float4 t = load_cols(T, ldt, u, q, F);
        acc.x += w * t.x;
        acc.y += w * t.y;
        acc.z += w * t.z;
        acc.w += w * t.w;
      }
    }
  }
#pragma unroll
  for (int d = LG; d < 64; d <<= 1) {
    acc.x += __shfl_xor(acc.x, d, 64);
    acc.y += __shfl_xor(acc.y, d, 64);
    acc.z += __shfl_xor(acc.z, d, 64);
    acc.w += __shfl_xor(acc.w, d, 64);
  }
  if (lane == 0) {
    stats[2 * v] = mx;
    stats[2 * v + 1] = inv;
  }
  if (lane >= LG || 4 * q >= F) return;
  const float ws = __expf(e_self - mx) * inv;
  const float4 t = load_cols(T, ldt, v, q, F);
  acc.x += ws * t.x;
  acc.y += ws * t.y;
  acc.z += ws * t.z;
  acc.w += ws * t.w;
  if (relu) {
    acc.x = fmaxf(acc.x, 0.f);
    acc.y = fmaxf(acc.y, 0.f);
    acc.z = fmaxf(acc.z, 0.f);
    acc.w = fmaxf(acc.w, 0.f);
  }
  store_cols(out, F, v, q, F, acc);
}

// Backward through the attention sum and the softmax for dst row v (one wave;
// the self edge is edge index c).  dT (stride ldt) and ds must be zero on
// entry; dT and ds_r gather atomics from every row.  dT may be null (the
// score gradients only).  dOut has row stride
// ld_do and is masked by mask > 0 (the layer's ReLU output) when given.
template <int LG>
__global__ void __launch_bounds__(kThreads)
attend_bwd_kernel(EdgeView b, const float* __restrict__ T, int32_t ldt, const float* __restrict__ s,
                  const float* __restrict__ stats, const float* __restrict__ dout, int64_t ld_do,
                  const float* __restrict__ mask, int32_t F, float* dT, float* ds) {
  constexpr int G = 64 / LG;
  const int lane = lane_id();
  const int g = lane / LG, q = lane % LG;
  const int64_t v = ((int64_t)blockIdx.x * kThreads + threadIdx.x) >> 6;
  if (v >= b.counts[0]) return;
  const int32_t e0 = b.indptr[v], c = b.indptr[v + 1] - e0;
  const int32_t ce = c + 1;  // with the self edge
  const float sl = s[2 * v], mx = stats[2 * v], inv = stats[2 * v + 1];
  const bool cols = 4 * q < F;
  float4 dO = make_float4(0.f, 0.f, 0.f, 0.f);
  if (cols) {
    dO = load_cols(dout, ld_do, v, q, F);
    if (mask) {
      const float4 mk = load_cols(mask, ld_do, v, q, F);
      dO.x = mk.x > 0.f ? dO.x : 0.f;
      dO.y = mk.y > 0.f ? dO.y : 0.f;
      dO.z = mk.z > 0.f ? dO.z : 0.f;
      dO.w = mk.w > 0.f ? dO.w : 0.f;
    }
  }
  auto edge = [&](int32_t l, int32_t* u, float* alpha, float* lk) {
    *u = l < c ? b.indices[e0 + l] : (int32_t)v;
    const float pre = sl + s[2 * *u + 1];
    *alpha = __expf(leaky(pre) - mx) * inv;
    *lk = pre > 0.f ? 1.f : kSlope;
  };
  float S = 0.f, P1 = 0.f, Q = 0.f;  // lanes q == 0 of each group
  for (int32_t base = 0; base < ce; base += 64) {
    const int32_t cc = ce - base < 64 ? ce - base : 64;
    int32_t my_u = 0;
    float my_a = 0.f, my_k = 0.f;
    if (lane < cc) edge(base + lane, &my_u, &my_a, &my_k);
    for (int32_t k = 0; k < cc; k += G) {
      const int32_t l = k + g;
      const int32_t u = __shfl(my_u, l & 63, 64);
      const float al = __shfl(my_a, l & 63, 64);
      const float lk = __shfl(my_k, l & 63, 64);
      const bool ok = l < cc;
      float d = 0.f;
      if (ok && cols) d = dot4(dO, load_cols(T, ldt, u, q, F));
#pragma unroll
      for (int x = 1; x < LG; x <<= 1) d += __shfl_xor(d, x, 64);
      if (dT && ok && cols) {
        float* o = dT + (int64_t)u * ldt + 4 * q;
        const float w[4] = {al * dO.x, al * dO.y, al * dO.z, al * dO.w};
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (4 * q + i < F) unsafeAtomicAdd(o + i, w[i]);
      }
      if (ok && q == 0) {
        S += al * d;
        P1 += al * lk * d;
        Q += al * lk;
        unsafeAtomicAdd(ds + 2 * (int64_t)u + 1, al * lk * d);
      }
    }
  }
  S = wave_sum(S);
  P1 = wave_sum(P1);
  Q = wave_sum(Q);
  if (lane == 0) ds[2 * v] = P1 - S * Q;
  // the -S_v alpha lk share of every edge's dpre
  for (int32_t l = lane; l < ce; l += 64) {
    int32_t u;
    float al, lk;
    edge(l, &u, &al, &lk);
    unsafeAtomicAdd(ds + 2 * (int64_t)u + 1, -S * al * lk);
  }
}

// dT_u += ds_r[u] a_r + [u < n_dst] ds_l[u] a_l for every src row u.
__global__ void __launch_bounds__(kThreads)
score_grad_kernel(const int32_t* counts, const float* __restrict__ a, int32_t F,
                  const float* __restrict__ ds, float* __restrict__ dT, int32_t ldt) {
  const int64_t n_src = counts[1], n_dst = counts[0];
  const int64_t total = n_src * F;
  for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * kThreads) {
    const int64_t u = i / F;
    const int32_t f = (int32_t)(i - u * F);
    float x = ds[2 * u + 1] * a[F + f];
    if (u < n_dst) x += ds[2 * u] * a[f];
    dT[u * ldt + f] += x;
  }
}

// [ds_l | ds_r]^T X in two passes: colsum_part_kernel<QL> gives each of its
// workgroups a chunk of rows (256 / QL row groups of QL lanes, a lane per
// 4-column chunk) and writes the chunk's two column sums to part[block]
// (2 x 256 floats; zeros for an empty chunk); colsum_final_kernel adds the
// parts in block order.  No atomics, and the result does not depend on timing.
constexpr int kColsumParts = 256;

template <int QL>
__global__ void __launch_bounds__(kThreads)
colsum_part_kernel(const int32_t* n_dev, int32_t cap, const float* __restrict__ w,
                   const float* __restrict__ X, int64_t ld, int32_t F, float* __restrict__ part) {
  constexpr int RG = kThreads / QL;
  __shared__ float4 red[2][RG][QL];
  int32_t n = *n_dev;
  n = n > cap ? cap : n;
  const int q = threadIdx.x % QL, rg = threadIdx.x / QL;
  const int64_t chunk = ((int64_t)n + gridDim.x - 1) / gridDim.x;
  const int64_t r0 = (int64_t)blockIdx.x * chunk;
  const int64_t r1 = r0 + chunk < n ? r0 + chunk : n;
  float4 a0 = make_float4(0.f, 0.f, 0.f, 0.f), a1 = a0;
  auto add = [&](float4 x, float w0, float w1) {
    a0.x += w0 * x.x;
    a0.y += w0 * x.y;
    a0.z += w0 * x.z;
    a0.w += w0 * x.w;
    a1.x += w1 * x.x;
    a1.y += w1 * x.y;
    a1.z += w1 * x.z;
    a1.w += w1 * x.w;
  };
  if (4 * q < F) {
    int64_t u = r0 + rg;
    // four rows in flight per lane
    for (; u + 3 * RG < r1; u += 4 * RG) {
      float4 x[4];
      float2 wv[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        x[i] = load_cols(X, ld, u + i * RG, q, F);
        wv[i] = reinterpret_cast<const float2*>(w)[u + i * RG];
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) add(x[i], wv[i].x, wv[i].y);
    }
    for (; u < r1; u += RG) {
      const float2 wv = reinterpret_cast<const float2*>(w)[u];
      add(load_cols(X, ld, u, q, F), wv.x, wv.y);
    }
  }
  red[0][rg][q] = a0;
  red[1][rg][q] = a1;
  __syncthreads();
  // thread t: column sum t of c = t / 256... one float per thread: 2 x 4 QL values
  for (int t = threadIdx.x; t < 2 * 4 * QL; t += kThreads) {
    const int c = t / (4 * QL), f = t % (4 * QL);
    float acc = 0.f;
    for (int g = 0; g < RG; ++g) {
      const float4 v = red[c][g][f / 4];
      acc += (f & 3) == 0 ? v.x : ((f & 3) == 1 ? v.y : ((f & 3) == 2 ? v.z : v.w));
    }
    part[(int64_t)blockIdx.x * 512 + c * 256 + f] = acc;
  }
}

// out[c * oc + f * of] = sum over the parts of part[b][c][f]: a wave per
// output, lane l over parts l, l + 64, ..., then a fixed-order wave sum.
__global__ void __launch_bounds__(kThreads)
colsum_final_kernel(const float* __restrict__ part, int32_t nparts, int32_t F, float* out, int64_t oc,
                    int64_t of) {
  const int lane = lane_id();
  const int64_t t = ((int64_t)blockIdx.x * kThreads + threadIdx.x) >> 6;
  if (t >= 2 * F) return;
  const int c = (int)(t / F), f = (int)(t % F);
  float acc = 0.f;
  for (int b = lane; b < nparts; b += 64) acc += part[(int64_t)b * 512 + c * 256 + f];
  acc = wave_sum(acc);
  if (lane == 0) out[c * oc + f * of] = acc;
}

inline int lanes_for(int32_t F) {
  int c = (F + 3) / 4, p = 1;
  while (p < c) p <<= 1;
  return p;
}

inline unsigned wave_grid(int64_t rows) {
  return (unsigned)std::max<int64_t>(1, ceil_div(rows * 64, kThreads));
}

inline unsigned stride_grid(int64_t n) {
  return (unsigned)std::min<int64_t>(4096, std::max<int64_t>(1, ceil_div(n, kThreads)));
}

int check_f(int32_t F, const char* who) {
  if (F < 1 || F > 256) return fail(GNN_EINVAL, "%s: width %d not in [1, 256]", who, F);
  return GNN_OK;
}

}  // namespace

int launch_gat_gather(const gnn_block* blk, const void* X, int32_t dtype, const int32_t* rows,
                      int64_t n_rows, int64_t ld_x, int32_t F, float* out, hipStream_t st) {
  if (blk->cap_src == 0) return GNN_OK;
  if (F % 4) return fail(GNN_EINVAL, "GAT gather: width %d not a multiple of 4", F);
  const int32_t c4 = F / 4;
  const unsigned grid = stride_grid((int64_t)blk->cap_src * c4);
  auto o = reinterpret_cast<float4*>(out);
  if (!rows) n_rows = INT64_MAX;
  if (dtype == GNN_F32)
    launch("gather", gather_kernel<GNN_F32>, grid, kThreads, 0, st, X, rows, n_rows, ld_x,
           (const int32_t*)blk->counts, blk->cap_src, c4, o);
  else
    launch("gather", gather_kernel<GNN_BF16>, grid, kThreads, 0, st, X, rows, n_rows, ld_x,
           (const int32_t*)blk->counts, blk->cap_src, c4, o);
  GNN_LAUNCH_CHECK("GAT gather");
  return GNN_OK;
}

int launch_gat_scores(const gnn_block* blk, const float* T, int32_t ldt, const float* a, int32_t F,
                      float* s, hipStream_t st) {
  if (blk->cap_src == 0) return GNN_OK;
  if (int rc = check_f(F, "GAT scores")) return rc;
  // 16 lanes per row (4 rows per wave), fewer for narrow rows
  const int lg = std::min(16, lanes_for(F));
  const unsigned grid = wave_grid(ceil_div((int64_t)blk->cap_src, 64 / lg));
  auto go = [&](auto kernel) {
    launch("gat_scores", kernel, grid, kThreads, 0, st, T, ldt, a, F, (const int32_t*)blk->counts, s);
  };
  switch (lg) {
    case 1: go(scores_kernel<1>); break;
    case 2: go(scores_kernel<2>); break;
    case 4: go(scores_kernel<4>); break;
    case 8: go(scores_kernel<8>); break;
    default: go(scores_kernel<16>); break;
  }
  GNN_LAUNCH_CHECK("GAT scores");
  return GNN_OK;
}

int launch_gat_attend(const gnn_block* blk, const float* T, int32_t ldt, const float* s, int32_t F,
                      int32_t relu, float* out, float* stats, hipStream_t st) {
  if (blk->cap_dst == 0) return GNN_OK;
  if (int rc = check_f(F, "GAT attention")) return rc;
  const EdgeView b{blk->indptr, blk->indices, blk->counts};
  const unsigned grid = wave_grid(blk->cap_dst);
  auto go = [&](auto kernel) {
    launch("gat_attend", kernel, grid, kThreads, 0, st, b, T, ldt, s, F, relu, out, stats);
  };
  switch (lanes_for(F)) {
    case 1: go(attend_kernel<1>); break;
    case 2: go(attend_kernel<2>); break;
    case 4: go(attend_kernel<4>); break;
    case 8: go(attend_kernel<8>); break;
    case 16: go(attend_kernel<16>); break;
    case 32: go(attend_kernel<32>); break;
    default: go(attend_kernel<64>); break;
  }
  GNN_LAUNCH_CHECK("GAT attention");
  return GNN_OK;
}

int launch_gat_attend_bwd(const gnn_block* blk, const float* T, int32_t ldt, const float* s,
                          const float* stats, const float* dout, int64_t ld_do, const float* mask,
                          int32_t F, float* dT, float* ds, hipStream_t st) {
  if (blk->cap_dst == 0) return GNN_OK;
  if (int rc = check_f(F, "GAT attention backward")) return rc;
  const EdgeView b{blk->indptr, blk->indices, blk->counts};
  const unsigned grid = wave_grid(blk->cap_dst);
  auto go = [&](auto kernel) {
    launch("gat_attend_bwd", kernel, grid, kThreads, 0, st, b, T, ldt, s, stats, dout, ld_do, mask,
           F, dT, ds);
  };
  switch (lanes_for(F)) {
    case 1: go(attend_bwd_kernel<1>); break;
    case 2: go(attend_bwd_kernel<2>); break;
    case 4: go(attend_bwd_kernel<4>); break;
    case 8: go(attend_bwd_kernel<8>); break;
    case 16: go(attend_bwd_kernel<16>); break;
    case 32: go(attend_bwd_kernel<32>); break;
    default: go(attend_bwd_kernel<64>); break;
  }
  GNN_LAUNCH_CHECK("GAT attention backward");
  return GNN_OK;
}

size_t gat_colsum_part_floats() { return (size_t)kColsumParts * 512; }

int launch_gat_colsum2(const int32_t* n_dev, int32_t cap, const float* w, const float* X, int64_t ld,
                       int32_t F, float* part, float* out, int64_t oc, int64_t of, hipStream_t st) {
  if (int rc = check_f(F, "GAT column sums")) return rc;
  const int ql = lanes_for(F);
  auto go = [&](auto kernel) {
    launch("gat_colsum", kernel, kColsumParts, kThreads, 0, st, n_dev, std::max(0, cap), w, X, ld, F,
           part);
  };
  switch (ql) {
    case 1: go(colsum_part_kernel<1>); break;
    case 2: go(colsum_part_kernel<2>); break;
    case 4: go(colsum_part_kernel<4>); break;
    case 8: go(colsum_part_kernel<8>); break;
    case 16: go(colsum_part_kernel<16>); break;
    case 32: go(colsum_part_kernel<32>); break;
    default: go(colsum_part_kernel<64>); break;
  }
  GNN_LAUNCH_CHECK("GAT column sums");
  launch("gat_colsum_final", colsum_final_kernel, wave_grid(2 * (int64_t)F), kThreads, 0, st,
         (const float*)part, (int32_t)kColsumParts, F, out, oc, of);
  GNN_LAUNCH_CHECK("GAT column sums");
  return GNN_OK;
}

int launch_gat_score_grad(const gnn_block* blk, const float* a, int32_t F, const float* ds, float* dT,
                          int32_t ldt, hipStream_t st) {
  if (blk->cap_src == 0) return GNN_OK;
  launch("gat_score_grad", score_grad_kernel, stride_grid((int64_t)blk->cap_src * F), kThreads, 0,
         st, (const int32_t*)blk->counts, a, F, ds, dT, ldt);
  GNN_LAUNCH_CHECK("GAT score gradient");
  return GNN_OK;
}

}  // namespace gnn
