// Output layer of the training step together with its loss (paper section
// 2.2, eq. (3), on the last layer of eq. (1)): for a tile of root rows,
//   Z  = X W                                   (logits, no activation)
//   l  = logsumexp(Z) - Z[y],  dZ = (softmax(Z) - onehot(y)) / B
//   dX = dZ W^T                                (input gradient)
//   dW = X^T dZ                                (weight gradient, per tile)
// in one launch.  With at most 64 classes each product is a few MFLOP per
// tile, so as separate launches they would be latency-bound and wait on each
// other; here one block keeps X, Z and dZ of its rows in LDS from the first
// product to the last.  The weight gradient is written per tile and summed in
// a fixed order by the SGD launch (no atomics, deterministic).
//
// Block: 8 waves, 16 rows.  fp32 MFMA 16x16x4: lane l feeds row/column l % 16
// and k-slot l / 16 of each operand; its accumulator holds rows 4 (l / 16) + r,
// column l % 16.  Extra blocks past the row tiles zero the rows of the input
// gradient that the following scatter accumulates into.
#include "internal.hpp"
#include "wave.hpp"

namespace gnn {

namespace {

constexpr int kThreads = 512;
constexpr int kWaves = kThreads / 64;
constexpr int R = kHeadRows;  // 16 rows per block
constexpr int KMAX = 512;     // layer input width: 2 x 256 (SAGE)
constexpr int CMAX = kHeadMaxClasses;
constexpr int ZS = CMAX + 4;  // LDS row stride of the logit and dZ tiles
constexpr int WS = CMAX + 4;  // LDS row stride of a wave's W slice (68 = 4 mod 16)
constexpr int kSpinLimit = 1 << 20;  // iterations of the bounded wait (about 0.1 s)
constexpr int64_t kMaxSplitBlocks = 1024;  // the split grid must be resident at once

inline int64_t padded_tiles(int32_t B) { return ceil_div(ceil_div(B, R), 8) * 8; }

typedef float floatx4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ floatx4 mfma(float a, float b, floatx4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

struct HeadArgs {
  HeadJob j;
  int32_t head_blocks;
  int* err;
};

// NT: 16-wide class tiles (C <= 16 NT); KB: the input width rounded up to
// 128, 256 or 512.  Wave w owns rows [w KW, (w + 1) KW) of W (KW = KB / 8):
// the k-slice of the forward product, the columns of dX and the rows of dW
// it computes.  It stages that slice in LDS once (16-byte loads of the
// contiguous rows) and reads both products' operands from there; X goes
// from global memory straight into registers.  Loops have static trip
// counts: padded k meets zero X values, padded classes zero dZ values, and
// padded outputs are never stored.
//
// SPLIT: the input width is cut into P = ceil(K / 128) parts of KB = 128 rows,
// one block per (row tile, part), so that every block stages a quarter of W
// at most; the P blocks of a row tile add their partial logits through an
// exchange buffer (device-scope atomic stores and loads; a block's stores
// are released by its arrival on the tile's counter, a release RMW after a
// barrier, and acquired by the bounded wait for all P arrivals before a
// barrier) and each then holds the full logits.  Block b
// takes tile (b / 8 / P) * 8 + b % 8, part b / 8 % P, so that the P blocks
// of a tile sit on one XCD (blocks are dealt to the 8 XCDs in turn).
template <int NT, int KB, bool SPLIT>
__global__ void __launch_bounds__(kThreads) head_kernel(HeadArgs ha) {
  constexpr int KW = KB / kWaves;  // W rows per wave
  constexpr int TPW = KW / 16;     // 16-wide tiles per wave (dX columns, dW rows)
  constexpr int CP = 16 * NT;      // padded classes
  const HeadJob& a = ha.j;
  const int tid = threadIdx.x;
  if ((int32_t)blockIdx.x >= ha.head_blocks) {
    // zero rows [lo, hi) of the input gradient that the scatter adds into
    const int32_t lo = a.zero_lo ? *a.zero_lo : 0;
    int32_t hi = *a.zero_hi;
    hi = hi > a.zero_cap ? a.zero_cap : hi;
    const int64_t c4 = a.zero_cols / 4, ld4 = a.zero_ld / 4;
    const int64_t n = lo < hi ? (int64_t)(hi - lo) * c4 : 0;
    const int64_t nb = (int64_t)gridDim.x - ha.head_blocks;
    float4* z = reinterpret_cast<float4*>(a.zero_p);
    for (int64_t i = ((int64_t)blockIdx.x - ha.head_blocks) * kThreads + tid; i < n; i += nb * kThreads)
      z[(lo + i / c4) * ld4 + i % c4] = make_float4(0.f, 0.f, 0.f, 0.f);
    return;
  }
  __shared__ __align__(16) float Wsl[kWaves * KW * WS];  // per wave: W slice, later its logits
  __shared__ __align__(16) float Zs[R * ZS];
  const int lane = tid & 63, w = tid >> 6;
  const int g = lane >> 4, c16 = lane & 15;
  const int K = a.K, C = a.C;
  int64_t tile = blockIdx.x;
  int part = 0, P = 1;
  if (SPLIT) {
    P = (K + KB - 1) / KB;
    const int64_t j = blockIdx.x >> 3;
    tile = (j / P) * 8 + (blockIdx.x & 7);
    part = (int)(j % P);
    if (tile * R >= a.B) return;  // a padding tile: its P blocks all leave
  }
  const int64_t row0 = tile * R;
  const int nr = (int64_t)a.B - row0 < R ? (int)((int64_t)a.B - row0) : R;
  const int k0 = part * KB + w * KW;  // first W row of this wave
  float* Wl = Wsl + w * KW * WS;

  // --- global reads, all issued before the first wait ---
  // W rows [k0, k0 + KW) x C: contiguous, read as float4 (rows past K: 0)
  constexpr int WV = (KW * CMAX / 4 + 63) / 64;  // float4 per lane at most
  const int n4 = K > k0 ? (min(K, k0 + KW) - k0) * C / 4 : 0;
  float4 wv[WV];
  const float4* Wg = reinterpret_cast<const float4*>(a.W + (int64_t)(n4 > 0 ? k0 : 0) * C);
#pragma unroll
  for (int i = 0; i < WV; ++i) {
    const int q = lane + 64 * i;
    wv[i] = Wg[q < n4 ? q : 0];
  }
  // forward A operand: X[c16][k0 + 16 m + 4 g + (0..3)] (step 4 m + i uses
  // k = k0 + 16 m + 4 g + i; the B operand follows the same order)
  float4 xa[KW / 16];
  {
    const bool rok = c16 < nr;
    const float4* xr = reinterpret_cast<const float4*>(a.X + (row0 + (rok ? c16 : 0)) * K);
#pragma unroll
    for (int m = 0; m < KW / 16; ++m) {
      const int k = k0 + 16 * m + 4 * g;
      const bool ok = rok && k < K;
      const float4 v = xr[ok ? k / 4 : 0];
      xa[m] = ok ? v : make_float4(0.f, 0.f, 0.f, 0.f);
    }
  }
  // dW A operand: X^T[k0 + 16 u + c16][4 s + g]
  float xt[TPW][R / 4];
#pragma unroll
  for (int u = 0; u < TPW; ++u)
#pragma unroll
    for (int s = 0; s < R / 4; ++s) {
      const int k = k0 + 16 * u + c16, r = 4 * s + g;
      const bool ok = r < nr && k < K;
      const float v = a.X[(row0 + (ok ? r : 0)) * K + (ok ? k : 0)];
      xt[u][s] = ok ? v : 0.f;
    }
  const int srow = tid >> 4, sq = tid & 15;
  int64_t li = -1;
  if (tid < R * 16 && srow < nr) li = a.label_rows ? a.label_rows[row0 + srow] : row0 + srow;

  // W slice into LDS (row stride WS; rows past K and padded classes: 0).
  // Element f = 4 q + t of the slice sits at row f / C, column f % C; the
  // lane's position advances by 256 elements per float4 step, and within a
  // float4 wraps to the next row at most once (C >= 4).
  {
    int c = (4 * lane) % C, addr = ((4 * lane) / C) * WS + c;
    const int dq = 256 / C, dr = 256 % C;
#pragma unroll
    for (int i = 0; i < WV; ++i) {
      const int q = lane + 64 * i;
      if (q < KW * C / 4) {
        const float4 v = q < n4 ? wv[i] : make_float4(0.f, 0.f, 0.f, 0.f);
        const float e[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int t = 0; t < 4; ++t) Wl[addr + t + (c + t >= C ? WS - C : 0)] = e[t];
      }
      c += dr;
      addr += dq * WS + dr;
      if (c >= C) {
        c -= C;
        addr += WS - C;
      }
    }
  }
  // padded classes [C, CP) of every row read as 0
  for (int f = lane; f < KW * 16; f += 64) {
    const int c = C + (f & 15);
    if (c < CP) Wl[(f >> 4) * WS + c] = 0.f;
  }
  __syncthreads();
  const int32_t y = (li >= 0 && li < a.n_labels) ? a.labels[li] : -1;

  // 1. partial logits over the wave's k-slice
  floatx4 acc[NT];
#pragma unroll
  for (int j = 0; j < NT; ++j) acc[j] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int m = 0; m < KW / 16; ++m) {
    const float xe[4] = {xa[m].x, xa[m].y, xa[m].z, xa[m].w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float* wr = Wl + (16 * m + 4 * g + i) * WS + c16;
#pragma unroll
      for (int j = 0; j < NT; ++j) acc[j] = mfma(xe[i], wr[16 * j], acc[j]);
    }
  }
  // dX operand (W^T[o][k0 + 16 u + c16], o = 4 s + g) into registers, then
  // the slice's memory takes this wave's partial logits
  float bt[TPW][CP / 4];
  if (a.dx0) {
#pragma unroll
    for (int u = 0; u < TPW; ++u)
#pragma unroll
      for (int s = 0; s < CP / 4; ++s) bt[u][s] = Wl[(16 * u + c16) * WS + 4 * s + g];
  }
  __syncthreads();  // (LDS reads of every wave done before any slice is overwritten)
#pragma unroll
  for (int j = 0; j < NT; ++j)
#pragma unroll
    for (int r = 0; r < 4; ++r) Wl[(4 * g + r) * ZS + 16 * j + c16] = acc[j][r];
  __syncthreads();

  // 2. softmax cross-entropy: 16 threads per row, 4 classes each
  float z[4] = {0.f, 0.f, 0.f, 0.f};
  if (tid < R * 16 && 4 * sq < CP) {
#pragma unroll
    for (int v = 0; v < kWaves; ++v) {
      const float4 p = *reinterpret_cast<const float4*>(&Wsl[v * KW * WS + srow * ZS + 4 * sq]);
      z[0] += p.x;
      z[1] += p.y;
      z[2] += p.z;
      z[3] += p.w;
    }
  }
  if (SPLIT && P > 1) {
    // exchange: this part's logits out, every part's in (in part order, so
    // that the P blocks of a tile hold bit-identical sums)
    float* xt_ = a.xch + tile * (int64_t)(kHeadMaxParts * R * CMAX);
    if (tid < R * 16 && 4 * sq < CP) {
#pragma unroll
      for (int e = 0; e < 4; ++e)
        __hip_atomic_store(&xt_[(part * R + srow) * CMAX + 4 * sq + e], z[e], __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
    }
    // every thread's exchange stores happen before the barrier, and the
    // arrival below releases them (release is cumulative)
    __syncthreads();
    int32_t* cnt = a.sync + 2 * tile;
    if (tid == 0) {
      __hip_atomic_fetch_add(cnt, 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
      int it = 0;
      while (__hip_atomic_load(cnt, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < P) {
        if (++it > kSpinLimit) {
          set_device_error(ha.err, GNN_DEVERR_SYNC);
          break;
        }
        __builtin_amdgcn_s_sleep(2);
      }
      // one acquire after the last read of the counter (fence synchronisation)
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    }
    // thread 0's acquire of all P arrivals, then the barrier: the other parts'
    // stores happen before every thread's exchange loads below
    __syncthreads();
    if (tid < R * 16 && 4 * sq < CP) {
#pragma unroll
      for (int e = 0; e < 4; ++e) z[e] = 0.f;
      for (int p = 0; p < P; ++p)
#pragma unroll
        for (int e = 0; e < 4; ++e)
          z[e] += __hip_atomic_load(&xt_[(p * R + srow) * CMAX + 4 * sq + e], __ATOMIC_RELAXED,
                                    __HIP_MEMORY_SCOPE_AGENT);
    }
    __syncthreads();
    if (tid == 0) {
      // the last part to have read resets the tile's counters for the next launch
      if (__hip_atomic_fetch_add(cnt + 1, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == P - 1) {
        __hip_atomic_store(cnt, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(cnt + 1, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
    }
  }
  if (tid < R * 16) {
    const int row = srow, q = sq;
    const bool live = row < nr;
    const int64_t gr = row0 + row;
    const bool ok = y >= 0 && y < C;
    float mx = -INFINITY;
#pragma unroll
    for (int e = 0; e < 4; ++e)
      if (4 * q + e < C) mx = fmaxf(mx, z[e]);
#pragma unroll
    for (int d = 8; d >= 1; d >>= 1) mx = fmaxf(mx, __shfl_xor(mx, d, 16));
    float ex[4], s = 0.f, zy = 0.f;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      ex[e] = 4 * q + e < C ? expf(z[e] - mx) : 0.f;
      s += ex[e];
      zy += 4 * q + e == y ? z[e] : 0.f;
    }
#pragma unroll
    for (int d = 8; d >= 1; d >>= 1) {
      s += __shfl_xor(s, d, 16);
      zy += __shfl_xor(zy, d, 16);
    }
    const float inv_s = 1.f / s, inv_b = 1.f / (float)a.B;
    float dz[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int c = 4 * q + e;
      dz[e] = (live && ok && c < C) ? (ex[e] * inv_s - (c == y ? 1.f : 0.f)) * inv_b : 0.f;
    }
    *reinterpret_cast<float4*>(&Zs[row * ZS + 4 * q]) = make_float4(dz[0], dz[1], dz[2], dz[3]);
    if (live && part == 0) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int c = 4 * q + e;
        if (c < C) {
          a.logits[gr * C + c] = z[e];
          a.dlogits[gr * C + c] = dz[e];
        }
      }
      if (q == 0) {
        a.row_loss[gr] = ok ? (logf(s) + mx - zy) : 0.f;
        if (!ok) set_device_error(ha.err, GNN_DEVERR_LABEL_RANGE);
      }
    }
  }
  __syncthreads();

  // 3. dX = dZ W^T for columns k0 + 16 u + c16
  if (a.dx0) {
    float za[CP / 4];
#pragma unroll
    for (int s = 0; s < CP / 4; ++s) za[s] = Zs[c16 * ZS + 4 * s + g];
#pragma unroll
    for (int u = 0; u < TPW; ++u) {
      floatx4 d = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < CP / 4; ++s) d = mfma(za[s], bt[u][s], d);
      const int col = k0 + 16 * u + c16;
      if (col < K) {
        float* base = col < a.split ? a.dx0 + col : a.dx1 + (col - a.split);
        const int64_t ld = col < a.split ? a.ld0 : a.ld1;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int row = 4 * g + r;
          if (row < nr) base[(row0 + row) * ld] = d[r];
        }
      }
    }
  }

  // 4. this tile's dW = X^T dZ (reduction over its 16 rows) for W rows
  //    k0 + 16 u + (0..15)
  {
    float zb[R / 4][NT];
#pragma unroll
    for (int s = 0; s < R / 4; ++s)
#pragma unroll
      for (int j = 0; j < NT; ++j) zb[s][j] = Zs[(4 * s + g) * ZS + 16 * j + c16];
    float* part_out = a.dw_part + tile * K * C;
#pragma unroll
    for (int u = 0; u < TPW; ++u) {
      floatx4 d[NT];
#pragma unroll
      for (int j = 0; j < NT; ++j) d[j] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < R / 4; ++s)
#pragma unroll
        for (int j = 0; j < NT; ++j) d[j] = mfma(xt[u][s], zb[s][j], d[j]);
#pragma unroll
      for (int j = 0; j < NT; ++j) {
        const int c = 16 * j + c16;
        if (c < C) {
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int k = k0 + 16 * u + 4 * g + r;
            if (k < K) part_out[(int64_t)k * C + c] = d[j][r];
          }
        }
      }
    }
  }
}

}  // namespace

int launch_head(const HeadJob& j, hipStream_t st) {
  if (j.B <= 0) return GNN_OK;
  if (j.K < 4 || j.K > KMAX || j.K % 4) return fail(GNN_EINVAL, "head: input width %d", j.K);
  if (j.C < 4 || j.C > CMAX) return fail(GNN_EINVAL, "head: %d classes not in [4, %d]", j.C, CMAX);
  if (!j.X || !j.W || !j.logits || !j.dlogits || !j.row_loss || !j.dw_part || !j.labels)
    return fail(GNN_EINVAL, "head: null pointer");
  if ((reinterpret_cast<uintptr_t>(j.X) | reinterpret_cast<uintptr_t>(j.W)) & 15)
    return fail(GNN_EINVAL, "head: X and W must be 16-byte aligned");
  if (j.dx0 && (!j.dx1 && j.split < j.K)) return fail(GNN_EINVAL, "head: dX split without a second part");
  const int64_t blocks = ceil_div(j.B, R);
  int64_t zblocks = 0;
  if (j.zero_p) {
    if (j.zero_ld % 4 || j.zero_cols % 4 || (reinterpret_cast<uintptr_t>(j.zero_p) & 15) || !j.zero_hi)
      return fail(GNN_EINVAL, "head: zeroed rows must be 16-byte aligned float4 rows");
    zblocks = std::min<int64_t>(1024, std::max<int64_t>(1, ceil_div((int64_t)j.zero_cap * (j.zero_cols / 4),
                                                                      kThreads * 4)));
  }
  const int nt = (j.C + 15) / 16;
  const int parts = (int)ceil_div(j.K, 128);
  // the split form: one block per (row tile, 128-row part of W), when there
  // is more than one part and the grid is resident at once
  const bool split = parts > 1 && j.xch && j.sync && padded_tiles(j.B) * parts <= kMaxSplitBlocks;
  const int64_t hblocks = split ? padded_tiles(j.B) * parts : blocks;
  HeadArgs ha{j, (int32_t)hblocks, device_error_word()};
  const dim3 grid((unsigned)(hblocks + zblocks));
  const int kb = j.K <= 128 ? 128 : (j.K <= 256 ? 256 : 512);
  auto go = [&](auto kernel) { launch("head", kernel, grid, kThreads, 0, st, ha); };
#define GNN_HEAD_CASE(N, KB_) \
  if (nt == N && kb == KB_) go(head_kernel<N, KB_, false>);
#define GNN_HEAD_CASES(N)                                                    \
  if (split) {                                                               \
    if (nt == N) go(head_kernel<N, 128, true>);                              \
  } else {                                                                   \
    GNN_HEAD_CASE(N, 128) GNN_HEAD_CASE(N, 256) GNN_HEAD_CASE(N, 512)        \
  }
  GNN_HEAD_CASES(1)
  GNN_HEAD_CASES(2)
  GNN_HEAD_CASES(3)
  GNN_HEAD_CASES(4)
#undef GNN_HEAD_CASES
#undef GNN_HEAD_CASE
  GNN_LAUNCH_CHECK("head");
  return GNN_OK;
}

int64_t head_part_elems(int32_t B, int32_t K, int32_t C) { return ceil_div(B, R) * (int64_t)K * C; }
int64_t head_xch_elems(int32_t B) { return padded_tiles(B) * kHeadMaxParts * R * CMAX; }
int64_t head_sync_words(int32_t B) { return 2 * padded_tiles(B); }

}  // namespace gnn
