// Layer-1 products of a step whose features are bf16 (the transformation
// step, paper section 2.1, with the bf16 operand rounding of the training
// step): the forward Z = X W and the weight gradient dW = X^T dZ, for the
// thin shapes of that layer -- tens of thousands of rows, at most 256 columns
// on each side -- where the generic tiled kernel re-reads operands and, for
// dW, pays for contended atomics.
//
// Forward: every workgroup rounds W to bf16 once and keeps W^T in LDS (rows of
// K + pad, conflict-free 16-byte reads); each wave then owns 32-row strips of
// X, which it loads straight from HBM into the MFMA operand layout (a lane's
// eight consecutive k values of one row are 16 contiguous bytes), and issues
// v_mfma_f32_32x32x16_bf16 (half the LDS bytes per flop of the 16x16 shape)
// with X as the first operand, so that one store writes 128 contiguous bytes
// of each of two output rows.  The wave index is made uniform, so the buffer
// resources stay scalar.
//
// Weight gradient: the reduction runs over the rows, which are the
// non-contiguous axis of both X and dZ.  A lane loads eight consecutive rows
// of four adjacent X columns and four adjacent dZ columns (8 bytes each) and
// transposes them in registers; lane c of a tile then supplies column 4c + t
// (X) or 4c + u (dZ), so tile (t, u) computes dW at rows 4i + t and columns
// 4j + u.  A workgroup owns a 128 x 64 output block over one chunk of rows;
// its eight waves (two per SIMD: one's loads are in flight while the other
// multiplies) each take a 64 x 64 half of the block and every fourth 32-row
// step, add their sums through LDS, and the workgroup writes one partial
// block.  The chunks' partials are summed by the optimizer launch (no
// atomics, a fixed order).  The chunks of an output block run on one XCD, so
// the X and dZ rows a chunk reads are shared in that XCD's L2.
#include "internal.hpp"
#include "wave.hpp"

namespace gnn {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kXcds = 8;

// Operand loads go through buffer resources: an offset at or past the
// resource's range reads as 0, so masked rows and columns cost no branch and
// the count of loads in flight stays static.
constexpr int32_t kBufWord3 = 0x00020000;  // raw untyped buffer (gfx9 family)
constexpr uint32_t kOob = 0x80000000u;     // past every range below

// Resource over `bytes` bytes from p (clamped to [0, 2^31 - 1]).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t bytes_rsrc(const void* p, int64_t bytes) {
  bytes = bytes < 0 ? 0 : (bytes > 0x7FFFFFFF ? 0x7FFFFFFF : bytes);
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, kBufWord3);
}

// Resource over `rows` rows of `ld` 16-bit elements from p (nothing if rows <= 0).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t rows_rsrc(const uint16_t* p, int64_t rows, int64_t ld) {
  return bytes_rsrc(p, rows * ld * 2);
}

__device__ __forceinline__ u32x4 load16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  const auto v = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
  return u32x4{(uint32_t)v[0], (uint32_t)v[1], (uint32_t)v[2], (uint32_t)v[3]};
}

__device__ __forceinline__ u32x2 load8(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  const auto v = __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, 0);
  return u32x2{(uint32_t)v[0], (uint32_t)v[1]};
}

// ---- forward ------------------------------------------------------------------
constexpr int kFwdThreads = 512;  // eight waves, two per SIMD
constexpr int kFwdWaves = kFwdThreads / 64;
constexpr int kFwdCols = 256;     // output columns staged (zeros past N)
constexpr int kFwdLds = 73728;    // bf16 elements of W^T (144 KiB)

template <int KS>
constexpr int fwd_kp() {
  return KS * 16 + 8;  // W^T row stride: 16-byte rows, conflict-free 16-byte reads
}
static_assert(kFwdCols == kThinFwdCols && fwd_kp<16>() == thin_fwd_kp(256) && fwd_kp<2>() == thin_fwd_kp(32),
              "the staged W^T layout written by a WtJob");

typedef float floatx16 __attribute__((ext_vector_type(16)));

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

// Z = X W (ReLU optional) for X [M x K] bf16 (row stride ldx), W [K x N] fp32
// (row stride ldw), Z fp32 (row stride ldo); K <= 16 KS, N <= 256, N % 4 ==
// 0.  Wave w of block b takes the 32-row strips 8 b + w, then + 8 * grid;
// v_mfma_f32_32x32x16_bf16 takes X (lane (g2, c32): row c32, k 16 ks + 8 g2
// .. + 7, 16 contiguous bytes) as the first operand and W^T from LDS as the
// second, so accumulator e of tile t holds Z[row 8 (e / 4) + 4 g2 + e % 4]
// [32 t + c32]: each store writes 128 contiguous bytes of two rows.  Every
// tile is computed (the staged W^T is zero past N), so the products carry no
// branches.  Blocks then do the fill ranges.  PRE: W^T is copied from wtg,
// written in this layout by an earlier launch (run_wt_job), instead of
// converted from W (every CU reads half the bytes from L2 and converts
// nothing: 19.2 -> 16.4 us for 36K rows of the 111M-node workload).
template <int KS, bool RELU, bool PRE>
__global__ void __launch_bounds__(kFwdThreads)
thin_fwd_kernel(const uint16_t* __restrict__ X, int64_t ldx, const float* __restrict__ W, int64_t ldw,
                const uint16_t* __restrict__ wtg, float* __restrict__ out, int64_t ldo, int32_t m_cap,
                const int32_t* m_dev, int32_t K, int32_t N, FillPair fills) {
  __shared__ __align__(16) uint16_t wt[kFwdLds];
  constexpr int KP = fwd_kp<KS>();
  static_assert(kFwdCols * KP <= kFwdLds, "W^T does not fit");
  const int32_t M = m_dev ? min(m_cap, *m_dev) : m_cap;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // uniform: scalar resources
  const int g2 = lane >> 5, c32 = lane & 31;
  const int64_t strips = ((int64_t)M + 31) >> 5;
  const int64_t sstride = (int64_t)gridDim.x * kFwdWaves;
  int64_t s = (int64_t)blockIdx.x * kFwdWaves + wave;

  // rows past M, and strips past the last, read as 0
  auto load_strip = [&](int64_t strip, u32x4 (&a)[KS]) {
    const int64_t row0 = strip * 32;
    const __amdgpu_buffer_rsrc_t r = rows_rsrc(X + (row0 < M ? row0 : 0) * ldx, M - row0, ldx);
    const uint32_t base = (uint32_t)((c32 * ldx + 8 * g2) * 2);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) a[ks] = load16(r, 16 * ks + 8 * g2 < K ? base + 32 * ks : kOob);
  };
  u32x4 a[KS];

  // W^T in LDS as bf16 (nearest even): job q covers k 8 kq .. + 7 and columns
  // 4 nq .. + 3; every load of a thread is issued before the first conversion.
  // The first strip's loads go out once W is staged: loads retire in issue
  // order, so issued first the strip's HBM reads held back the conversion of
  // W, which the L2 serves (19.5 -> 19.0 us for 36K rows of the 111M-node
  // workload)
  if constexpr (PRE) {
    constexpr int kChunks = kFwdCols * KP / 8;
    constexpr int kPer = (kChunks + kFwdThreads - 1) / kFwdThreads;
    const uint4* src = reinterpret_cast<const uint4*>(wtg);
    uint4* dst = reinterpret_cast<uint4*>(wt);
    uint4 r[kPer];
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      const int q = threadIdx.x + j * kFwdThreads;
      r[j] = q < kChunks ? src[q] : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      const int q = threadIdx.x + j * kFwdThreads;
      if (q < kChunks) dst[q] = r[j];
    }
  } else {
    constexpr int kNq = kFwdCols / 4, kJobs = KS * 2 * kNq;
    constexpr int kPer = (kJobs + kFwdThreads - 1) / kFwdThreads;
    const __amdgpu_buffer_rsrc_t rw = bytes_rsrc(W, (int64_t)K * ldw * 4);
    u32x4 r[kPer][8];
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      const int q = threadIdx.x + j * kFwdThreads;
      const int kq = q / kNq, n0 = 4 * (q % kNq);
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int k = 8 * kq + i;
        r[j][i] = load16(rw, (q < kJobs && k < K && n0 < N) ? (uint32_t)(((int64_t)k * ldw + n0) * 4) : kOob);
      }
    }
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      const int q = threadIdx.x + j * kFwdThreads;
      if (q >= kJobs) continue;
      const int k0 = 8 * (q / kNq), n0 = 4 * (q % kNq);
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        bf16x8 v;
#pragma unroll
        for (int i = 0; i < 8; ++i) v[i] = (__bf16)__uint_as_float(r[j][i][c]);
        *reinterpret_cast<bf16x8*>(&wt[(n0 + c) * KP + k0]) = v;
      }
    }
  }
  __builtin_amdgcn_sched_barrier(0);  // (keeps the strip's loads after W's)
  load_strip(s, a);
  __syncthreads();

  for (; s < strips; s += sstride) {
    floatx16 acc[kFwdCols / 32];
#pragma unroll
    for (int t = 0; t < kFwdCols / 32; ++t)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[t][e] = 0.f;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const uint16_t* wrow = &wt[c32 * KP + 16 * ks + 8 * g2];
#pragma unroll
      for (int t = 0; t < kFwdCols / 32; ++t) {
        const bf16x8 bv = *reinterpret_cast<const bf16x8*>(wrow + 32 * t * KP);
        acc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(a[ks]), bv, acc[t], 0, 0, 0);
      }
    }
    const int64_t next = s + sstride;
    if (next < strips) load_strip(next, a);
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int64_t row = s * 32 + 8 * (e / 4) + 4 * g2 + (e % 4);
      if (row < M) {
        float* o = out + row * ldo + c32;
#pragma unroll
        for (int t = 0; t < kFwdCols / 32; ++t)
          if (32 * t + c32 < N) o[32 * t] = RELU ? fmaxf(acc[t][e], 0.f) : acc[t][e];
      }
    }
  }
  run_fills(fills, blockIdx.x, gridDim.x, kFwdThreads);
}

// ---- weight gradient -----------------------------------------------------------
constexpr int kDwThreads = 512;              // eight waves, two per SIMD
constexpr int kDwRows = 128, kDwCols = 64;   // output block of a workgroup
constexpr int kDwMaxParts = 32;

// rows 8 g + r (r = 0..7) of a 32-row step: four X columns and four dZ
// columns (8 bytes each)
struct DwRegs {
  u32x2 x[8];
  u32x2 z[8];
};

// X^T dZ over rows [m_lo, m_hi) into per-chunk partials part[c][kw x N].
// Wave w: half h = w & 1 of the block's X columns (64 each), phase w >> 1 of
// the 32-row steps.  Grid: ceil(nparts / 8) * 8 * (output blocks) workgroups.
__global__ void __launch_bounds__(kDwThreads)
thin_dw_kernel(const uint16_t* __restrict__ X, int64_t ldx, const uint16_t* __restrict__ Z, int64_t ldz,
               int32_t m_cap, const int32_t* m_dev, int32_t kw, int32_t N, float* __restrict__ part,
               int32_t nparts) {
  __shared__ __align__(16) float red[kDwRows * kDwCols];
  const int32_t M = m_dev ? min(m_cap, *m_dev) : m_cap;
  const int nbk = (kw + kDwRows - 1) / kDwRows, nbn = (N + kDwCols - 1) / kDwCols;
  const int nob = nbk * nbn;
  const int b = blockIdx.x, xcd = b % kXcds, idx = b / kXcds;
  const int c = (idx / nob) * kXcds + xcd, o = idx % nob;
  if (c >= nparts) return;
  const int kb = o / nbn, nb = o - kb * nbn;
  int32_t chunk = (M + nparts - 1) / nparts;
  chunk = (chunk + 31) & ~31;
  const int32_t m_lo = min(M, c * chunk), m_hi = min(M, m_lo + chunk);

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // uniform: scalar resources
  const int half = wave & 1, phase = wave >> 1;
  const int g = lane >> 4, c16 = lane & 15;
  const int32_t xc = kb * kDwRows + 64 * half + 4 * c16;  // first X column of the lane
  const int32_t zc = nb * kDwCols + 4 * c16;              // first dZ column of the lane
  const bool xok = xc < kw, zok = zc < N;

  auto load = [&](int32_t m0, DwRegs& R) {
    const int32_t b0 = m0 < m_hi ? m0 : m_lo;
    const __amdgpu_buffer_rsrc_t rx = rows_rsrc(X + (int64_t)b0 * ldx, m_hi - m0, ldx);
    const __amdgpu_buffer_rsrc_t rz = rows_rsrc(Z + (int64_t)b0 * ldz, m_hi - m0, ldz);
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      const uint32_t rr = (uint32_t)(8 * g + r);
      R.x[r] = load8(rx, xok ? (uint32_t)((rr * ldx + xc) * 2) : kOob);
      R.z[r] = load8(rz, zok ? (uint32_t)((rr * ldz + zc) * 2) : kOob);
    }
  };

  floatx4 acc[4][4];
#pragma unroll
  for (int t = 0; t < 4; ++t)
#pragma unroll
    for (int u = 0; u < 4; ++u) acc[t][u] = floatx4{0.f, 0.f, 0.f, 0.f};

  // element (row r, column t) of 16-bit pairs: half t & 1 of word t >> 1
  auto tr4 = [&](const u32x2 (&v)[8], bf16x8 (&o)[4]) {
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      u32x4 w;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const uint32_t lo = v[2 * e][t >> 1], hi = v[2 * e + 1][t >> 1];
        w[e] = (t & 1) ? ((lo >> 16) | (hi & 0xFFFF0000u)) : ((lo & 0xFFFFu) | (hi << 16));
      }
      o[t] = as_bf16x8(w);
    }
  };
  auto step = [&](const DwRegs& R) {
    bf16x8 xa[4], zb[4];
    tr4(R.x, xa);
    tr4(R.z, zb);
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int u = 0; u < 4; ++u)
        acc[t][u] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xa[t], zb[u], acc[t][u], 0, 0, 0);
  };

  // phase p takes the 32-row steps p, p + 4, ...; the next step's loads in flight
  constexpr int32_t kStride = 32 * 4;
  DwRegs R0, R1;
  int32_t m0 = m_lo + 32 * phase;
  load(m0, R0);
  while (m0 < m_hi) {
    load(m0 + kStride, R1);
    step(R0);
    m0 += kStride;
    if (m0 >= m_hi) break;
    load(m0 + kStride, R0);
    step(R1);
    m0 += kStride;
  }

  // lane (g, c16) holds, for tile (t, u) and accumulator q, dW at local row
  // 64 half + 16 g + 4 q + t and local column 4 c16 + u; the four phases add
  // their sums in LDS in phase order (the halves write disjoint rows), the
  // last one adds its own and stores the partial
  float* dst = part + (int64_t)c * kw * N;
  for (int p = 0; p < 4; ++p) {
    if (phase == p) {
#pragma unroll
      for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int lr = 64 * half + 16 * g + 4 * q + t;
          float4 v = make_float4(acc[t][0][q], acc[t][1][q], acc[t][2][q], acc[t][3][q]);
          float4* l = reinterpret_cast<float4*>(&red[lr * kDwCols + 4 * c16]);
          if (p > 0) {
            const float4 s = *l;
            v = make_float4(s.x + v.x, s.y + v.y, s.z + v.z, s.w + v.w);
          }
          if (p < 3) {
            *l = v;
          } else {
            const int32_t row = kb * kDwRows + lr;
            if (row < kw && zok) *reinterpret_cast<float4*>(dst + (int64_t)row * N + zc) = v;
          }
        }
    }
    if (p < 3) __syncthreads();
  }
}

template <int KS>
void launch_fwd_ks(const char* name, bool relu, unsigned grid, const uint16_t* X, int64_t ldx,
                   const float* W, int64_t ldw, const uint16_t* wt, float* out, int64_t ldo,
                   int32_t m_cap, const int32_t* m_dev, int32_t K, int32_t N, const FillPair& fills,
                   hipStream_t st) {
  auto go = [&](auto kernel) {
    launch(name, kernel, dim3(grid), kFwdThreads, 0, st, X, ldx, W, ldw, wt, out, ldo, m_cap, m_dev, K,
           N, fills);
  };
  if (wt) {
    if (relu) go(thin_fwd_kernel<KS, true, true>);
    else go(thin_fwd_kernel<KS, false, true>);
  } else {
    if (relu) go(thin_fwd_kernel<KS, true, false>);
    else go(thin_fwd_kernel<KS, false, false>);
  }
}

// 16-wide k steps of the instance that takes K (0: none)
int fwd_ks(int32_t K) { return thin_fwd_ks(K); }

bool aligned(const void* p, int bytes) { return (reinterpret_cast<uintptr_t>(p) & (uintptr_t)(bytes - 1)) == 0; }

}  // namespace

bool thin_fwd_ok(const uint16_t* X, int64_t ldx, const float* W, int64_t ldw, const float* out,
                 int64_t ldo, int32_t K, int32_t N) {
  const int ks = fwd_ks(K);
  return ks > 0 && K > 0 && K % 8 == 0 && N > 0 && N % 4 == 0 && N <= kFwdCols && ldx >= K && ldx % 8 == 0 &&
         ldw >= N && ldw % 4 == 0 && ldo >= N && ldo % 4 == 0 && aligned(X, 16) && aligned(W, 16) &&
         aligned(out, 16);
}

int launch_thin_fwd(const uint16_t* X, int64_t ldx, const float* W, int64_t ldw, float* out,
                    int64_t ldo, int32_t m_cap, const int32_t* m_dev, int32_t K, int32_t N, bool relu,
                    const FillPair& fills, const char* name, hipStream_t st, const uint16_t* wt) {
  if (!thin_fwd_ok(X, ldx, W, ldw, out, ldo, K, N))
    return fail(GNN_EINVAL, "thin forward: unsupported shape or alignment");
  if (wt && !aligned(wt, 16)) return fail(GNN_EINVAL, "thin forward: staged W^T not 16-byte aligned");
  if (m_cap <= 0) {
    FillRange fr[2];
    int n = 0;
    for (int r = 0; r < 2; ++r)
      if (fills.n[r] > 0) fr[n++] = FillRange{fills.p[r], fills.n[r], fills.v[r]};
    return launch_fill(fr, n, st);
  }
  // one workgroup per CU (the staged W^T takes most of the LDS), never more
  // than the strips need
  const int64_t strips = ceil_div(m_cap, 32);
  int64_t grid = std::min<int64_t>(device_cu_count(), ceil_div(strips, kFwdWaves));
  grid = std::max<int64_t>(grid, std::max<int64_t>(1, fill_blocks(fills, kFwdThreads)));
  switch (fwd_ks(K)) {
    case 2: launch_fwd_ks<2>(name, relu, (unsigned)grid, X, ldx, W, ldw, wt, out, ldo, m_cap, m_dev, K, N, fills, st); break;
    case 4: launch_fwd_ks<4>(name, relu, (unsigned)grid, X, ldx, W, ldw, wt, out, ldo, m_cap, m_dev, K, N, fills, st); break;
    case 8: launch_fwd_ks<8>(name, relu, (unsigned)grid, X, ldx, W, ldw, wt, out, ldo, m_cap, m_dev, K, N, fills, st); break;
    default: launch_fwd_ks<16>(name, relu, (unsigned)grid, X, ldx, W, ldw, wt, out, ldo, m_cap, m_dev, K, N, fills, st); break;
  }
  GNN_LAUNCH_CHECK("thin forward");
  return GNN_OK;
}

int32_t thin_dw_parts(int32_t m_cap) {
  // chunks of at least 512 rows, at most kDwMaxParts, a multiple of 8 (whole
  // XCD rounds)
  int64_t p = ceil_div(std::max<int32_t>(m_cap, 1), 512);
  p = std::min<int64_t>(kDwMaxParts, ceil_div(p, kXcds) * kXcds);
  return (int32_t)p;
}

bool thin_dw_ok(const uint16_t* X, int64_t ldx, const uint16_t* Z, int64_t ldz, int32_t kw, int32_t N) {
  return kw > 0 && kw % 4 == 0 && N > 0 && N % 4 == 0 && ldx >= kw && ldx % 4 == 0 && ldz >= N &&
         ldz % 4 == 0 && aligned(X, 8) && aligned(Z, 8);
}

int launch_thin_dw(const uint16_t* X, int64_t ldx, const uint16_t* Z, int64_t ldz, int32_t m_cap,
                   const int32_t* m_dev, int32_t kw, int32_t N, float* part, int32_t nparts,
                   const char* name, hipStream_t st) {
  if (!thin_dw_ok(X, ldx, Z, ldz, kw, N) || !part || nparts < 1 || nparts > kDwMaxParts ||
      !aligned(part, 16))
    return fail(GNN_EINVAL, "thin weight gradient: unsupported shape or alignment");
  const int64_t nob = ceil_div(kw, kDwRows) * ceil_div(N, kDwCols);
  const int64_t grid = ceil_div(nparts, kXcds) * kXcds * nob;
  if (grid > INT32_MAX / 2) return fail(GNN_EINVAL, "thin weight gradient: grid too large");
  launch(name, thin_dw_kernel, dim3((unsigned)grid), kDwThreads, 0, st, X, ldx, Z, ldz,
         std::max<int32_t>(m_cap, 0), m_dev, kw, N, part, nparts);
  GNN_LAUNCH_CHECK("thin weight gradient");
  return GNN_OK;
}

}  // namespace gnn
