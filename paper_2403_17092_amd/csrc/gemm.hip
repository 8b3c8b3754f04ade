// Dense update GEMMs of a layer (the transformation step, paper section 2.1):
// forward Z = [H_dst | agg] [W_self; W_neigh] (GraphSAGE) or agg W (GCN),
// backward dW = X^T dZ (split over rows, atomically reduced) and dX = dZ W^T.
//
// One kernel serves every case through "views": a logical operand is one or
// two row-major matrices joined along rows or columns, optionally read
// transposed, fp32 or bf16.  The tile loop uses the fp32 matrix cores:
// v_mfma_f32_16x16x4_f32, 64 x 64 x 16 block tiles, four wave64s each owning
// a 32 x 32 sub-tile (2 x 2 MFMA tiles), operands staged through LDS in
// k-major order with a register prefetch of the next k-slab.
#include "internal.hpp"
#include "wave.hpp"

namespace gnn {

namespace {

constexpr int BM = 64, BN = 64, BK = 16;
constexpr int kThreads = 256;
constexpr int PAD = 4;

typedef float floatx4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf16_to_f32(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

// Element (i, j) of a logical view (caller guarantees it is in range).
__device__ __forceinline__ float view_load(const MatView& v, int64_t i, int64_t j) {
  if (v.trans) {
    const int64_t t = i;
    i = j;
    j = t;
  }
  const bool second = v.axis == 0 ? (i >= v.split) : (j >= v.split);
  if (second) {
    if (v.axis == 0) i -= v.split;
    else j -= v.split;
  }
  const void* p = second ? v.p1 : v.p0;
  const int64_t ld = second ? v.ld1 : v.ld0;
  const int32_t dt = second ? v.dtype1 : v.dtype0;
  const int64_t off = i * ld + j;
  return dt == GNN_F32 ? static_cast<const float*>(p)[off]
                       : bf16_to_f32(static_cast<const uint16_t*>(p)[off]);
}

__device__ __forceinline__ void out_store(const OutView& o, int64_t i, int64_t j, float x,
                                          int epilogue) {
  const bool second = o.axis == 0 ? (i >= o.split) : (j >= o.split);
  if (second) {
    if (o.axis == 0) i -= o.split;
    else j -= o.split;
  }
  float* p = (second ? o.p1 : o.p0) + i * (second ? o.ld1 : o.ld0) + j;
  if (epilogue == 2) {
    unsafeAtomicAdd(p, x);
  } else {
    *p = epilogue == 1 ? fmaxf(x, 0.f) : x;
  }
}

__global__ void __launch_bounds__(kThreads)
gemm_kernel(MatView A, MatView B, OutView C, int32_t m_cap, int32_t N, int32_t k_cap,
            const int32_t* m_dev, const int32_t* k_dev, int32_t k_chunk, int32_t epilogue) {
  __shared__ float As[BK][BM + PAD];
  __shared__ float Bs[BK][BN + PAD];

  int32_t M = m_cap, K = k_cap;
  if (m_dev) M = min(M, *m_dev);
  if (k_dev) K = min(K, *k_dev);
  const int64_t m0 = (int64_t)blockIdx.x * BM;
  const int64_t n0 = (int64_t)blockIdx.y * BN;
  if (m0 >= M) return;
  const int32_t kbeg = blockIdx.z * k_chunk;
  const int32_t kend = min(K, kbeg + k_chunk);
  if (kbeg >= kend) return;

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = (wave >> 1) * 32, wn = (wave & 1) * 32;

  floatx4 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};

  // loader mappings: coalesce along the contiguous physical axis
  float ra[4], rb[4];
  auto load_tiles = [&](int32_t k0) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int e = tid + kThreads * r;
      int mi, ki;
      if (A.trans) {
        mi = e & (BM - 1);
        ki = e / BM;
      } else {
        mi = e / BK;
        ki = e & (BK - 1);
      }
      const int64_t gm = m0 + mi, gk = (int64_t)k0 + ki;
      ra[r] = (gm < M && gk < kend) ? view_load(A, gm, gk) : 0.f;
      int ni, kj;
      if (B.trans) {
        ni = e / BK;
        kj = e & (BK - 1);
      } else {
        ni = e & (BN - 1);
        kj = e / BN;
      }
      const int64_t gn = n0 + ni, gk2 = (int64_t)k0 + kj;
      rb[r] = (gn < N && gk2 < kend) ? view_load(B, gk2, gn) : 0.f;
    }
  };
  auto store_tiles = [&]() {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int e = tid + kThreads * r;
      if (A.trans) As[e / BM][e & (BM - 1)] = ra[r];
      else As[e & (BK - 1)][e / BK] = ra[r];
      if (B.trans) Bs[e & (BK - 1)][e / BK] = rb[r];
      else Bs[e / BN][e & (BN - 1)] = rb[r];
    }
  };

  load_tiles(kbeg);
  for (int32_t k0 = kbeg; k0 < kend; k0 += BK) {
    __syncthreads();
    store_tiles();
    __syncthreads();
    if (k0 + BK < kend) load_tiles(k0 + BK);
#pragma unroll
    for (int kk = 0; kk < BK; kk += 4) {
      const int kr = kk + (lane >> 4);
      const int c = lane & 15;
      const float a0 = As[kr][wm + c];
      const float a1 = As[kr][wm + 16 + c];
      const float b0 = Bs[kr][wn + c];
      const float b1 = Bs[kr][wn + 16 + c];
      acc[0][0] = __builtin_amdgcn_mfma_f32_16x16x4f32(a0, b0, acc[0][0], 0, 0, 0);
      acc[0][1] = __builtin_amdgcn_mfma_f32_16x16x4f32(a0, b1, acc[0][1], 0, 0, 0);
      acc[1][0] = __builtin_amdgcn_mfma_f32_16x16x4f32(a1, b0, acc[1][0], 0, 0, 0);
      acc[1][1] = __builtin_amdgcn_mfma_f32_16x16x4f32(a1, b1, acc[1][1], 0, 0, 0);
    }
  }

  // D layout of 16x16x4: lane l holds rows 4*(l/16) + r, column l%16
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t gm = m0 + wm + 16 * i + 4 * (lane >> 4) + r;
        const int64_t gn = n0 + wn + 16 * j + (lane & 15);
        if (gm < M && gn < N) out_store(C, gm, gn, acc[i][j][r], epilogue);
      }
}

}  // namespace

int launch_gemm(const MatView& A, const MatView& B, const OutView& C, int32_t m_cap, int32_t N,
                int32_t k_cap, const int32_t* m_dev, const int32_t* k_dev, int32_t epilogue,
                hipStream_t st) {
  if (m_cap <= 0 || N <= 0 || k_cap <= 0) return GNN_OK;
  const int64_t gm = ceil_div(m_cap, BM), gn = ceil_div(N, BN);
  int32_t k_chunk = k_cap;
  int64_t gz = 1;
  if (epilogue == 2) {
    // split the reduction so the grid has enough blocks to fill the GPU
    const int64_t want = std::max<int64_t>(1, 1024 / (gm * gn));
    k_chunk = (int32_t)std::max<int64_t>(256, ceil_div(ceil_div(k_cap, want), BK) * BK);
    gz = ceil_div(k_cap, k_chunk);
  }
  if (gz > 65535 || gn > 65535) return fail(GNN_EINVAL, "gemm: grid too large");
  gemm_kernel<<<dim3((unsigned)gm, (unsigned)gn, (unsigned)gz), kThreads, 0, st>>>(
      A, B, C, m_cap, N, k_cap, m_dev, k_dev, k_chunk, epilogue);
  GNN_LAUNCH_CHECK("gemm");
  return GNN_OK;
}

}  // namespace gnn
