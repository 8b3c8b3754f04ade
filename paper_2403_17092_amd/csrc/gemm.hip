// Dense update GEMMs of a layer (the transformation step, paper section 2.1):
// forward Z = X W with X = [H_dst | agg] (GraphSAGE) or agg (GCN) and W the
// stacked layer weights, backward dW = X^T dZ (split over rows, atomically
// reduced) and dX = dZ W^T.
//
// Tiling for CDNA4: 64 x 64 x 32 block tiles, 256 threads = four wave64s, each
// owning a 32 x 32 sub-tile computed with v_mfma_f32_16x16x4_f32 (2 x 2 MFMA
// tiles).  Operands are staged through double-buffered LDS; the next k-slab is
// loaded into registers while the current one feeds the matrix cores, so one
// barrier per slab suffices.  Global loads are 128-bit along each operand's
// contiguous axis, and every per-thread address is a fixed base plus a
// uniform per-slab stride.  Block ids are remapped so that the blocks sharing
// an A tile run on the same XCD (shared L2).  Split-K (atomic epilogue) sizes
// its chunks from the live reduction length read on the device.
#include "internal.hpp"
#include "wave.hpp"

namespace gnn {

namespace {

constexpr int BM = 64, BN = 64, BK = 32;
constexpr int kThreads = 256;
constexpr int kXcds = 8;
constexpr int H = BK / 16;   // staged 4-vectors per thread per operand per slab
constexpr int KQ = BK / 4;   // 4-vectors along k in one row of a slab

typedef float floatx4 __attribute__((ext_vector_type(4)));

struct Operand {
  const float* p;
  int64_t ld;
  int32_t vec;  // 128-bit loads allowed
};

struct Out {
  float* p0;
  float* p1;
  int64_t ld0, ld1;
  int32_t split, axis;
};

__device__ __forceinline__ void out_store(const Out& o, int64_t i, int64_t j, float x, int epilogue) {
  const bool second = o.axis == 0 ? (i >= o.split) : (j >= o.split);
  if (second) {
    if (o.axis == 0) i -= o.split;
    else j -= o.split;
  }
  float* p = (second ? o.p1 : o.p0) + i * (second ? o.ld1 : o.ld0) + j;
  if (epilogue == 2) unsafeAtomicAdd(p, x);
  else *p = epilogue == 1 ? fmaxf(x, 0.f) : x;
}

// Four consecutive elements p[off .. off+3]; elements whose column (c + e) is
// at or past c_lim, or all of them when !valid, read as 0 (from a clamped,
// in-bounds address).  VEC needs c and c_lim to be multiples of 4, so a chunk
// is entirely valid or not.
template <bool VEC>
__device__ __forceinline__ float4 load4(const float* __restrict__ p, int64_t off, bool valid,
                                        int64_t c, int64_t c_lim) {
  if (VEC) {
    valid = valid && c < c_lim;
    const float4 x = *reinterpret_cast<const float4*>(p + (valid ? off : 0));
    return valid ? x : make_float4(0.f, 0.f, 0.f, 0.f);
  }
  float v[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const bool ve = valid && (c + e) < c_lim;
    const float x = p[ve ? off + e : 0];
    v[e] = ve ? x : 0.f;
  }
  return make_float4(v[0], v[1], v[2], v[3]);
}

// AT / BT: operand read transposed (A^T: physical [k][m]; B^T: physical [n][k]).
// AV / BV: 128-bit loads allowed.
//
// LDS layout per operand follows its contiguous global axis, so staging is a
// plain copy: a k-contiguous operand (A, or B^T) is held as [row][k] with rows
// padded to keep 16-byte alignment and read with 128-bit LDS loads; a
// row-contiguous operand (A^T, or B) is held as [k][row] with an odd stride
// (conflict-free scalar access).  Within a slab, lane group g = lane / 16
// contributes k = g * KQ + j to MFMA step j; the same permutation on both
// operands leaves the dot products unchanged and makes each lane's k-values of
// a row contiguous.
template <bool AT, bool BT, bool AV, bool BV>
__global__ void __launch_bounds__(kThreads)
gemm_kernel(Operand A, Operand B, Out C, int32_t m_cap, int32_t N, int32_t k_cap,
            const int32_t* m_dev, const int32_t* k_dev, int32_t epilogue, int32_t min_chunk) {
  constexpr bool AROW = !AT, BROW = BT;   // [row][k] layouts
  constexpr int KPR = BK + 4;             // row-layout stride
  constexpr int KPC = BM + 1;             // column-layout stride (BM == BN)
  constexpr int AE = AROW ? BM * KPR : BK * KPC;
  constexpr int BE = BROW ? BN * KPR : BK * KPC;
  __shared__ __align__(16) float As[2][AE];
  __shared__ __align__(16) float Bs[2][BE];

  int32_t M = m_cap, K = k_cap;
  if (m_dev) M = min(M, *m_dev);
  if (k_dev) K = min(K, *k_dev);

  // XCD-aware tile order: consecutive block ids go to consecutive XCDs, so
  // m-tile mt is owned by XCD mt % 8 and its n-tiles are consecutive blocks of
  // that XCD (they share the A tile in that XCD's L2).  Live rows below the
  // capacity still spread over all XCDs.
  const int gn = (N + BN - 1) / BN;
  const int b = blockIdx.x;
  const int xcd = b % kXcds, idx = b / kXcds;
  const int64_t mt = (int64_t)(idx / gn) * kXcds + xcd;
  const int64_t m0 = mt * BM;
  const int64_t n0 = (int64_t)(idx % gn) * BN;
  if (m0 >= M) return;

  // split-K over the live reduction length
  int32_t kbeg = 0, kend = K;
  if (gridDim.z > 1) {
    int32_t parts = (K + min_chunk - 1) / min_chunk;
    parts = parts < 1 ? 1 : (parts > (int32_t)gridDim.z ? (int32_t)gridDim.z : parts);
    if ((int32_t)blockIdx.z >= parts) return;
    int32_t chunk = (K + parts - 1) / parts;
    chunk = (chunk + BK - 1) / BK * BK;
    kbeg = blockIdx.z * chunk;
    kend = min(K, kbeg + chunk);
    if (kbeg >= kend) return;
  }

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = (wave >> 1) * 32, wn = (wave & 1) * 32;
  const int g = lane >> 4, c16 = lane & 15;

  floatx4 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};

  // Staged 4-vector h of each operand: a k-contiguous operand takes (row
  // t / KQ, k (t % KQ) * 4), a row-contiguous one (k t / 16, row (t % 16) * 4).
  // Per thread: the offset at the first slab, the k coordinate at the first
  // slab, the fixed coordinate (row or column) and its validity.
  int64_t aoff[H], boff[H];
  int32_t ak[H], bk[H];
  int64_t afix[H], bfix[H];
  bool aok[H], bok[H];
#pragma unroll
  for (int h = 0; h < H; ++h) {
    const int t = tid + kThreads * h;
    if (AROW) {
      afix[h] = m0 + t / KQ;
      ak[h] = kbeg + (t % KQ) * 4;
      aok[h] = afix[h] < M;
      aoff[h] = afix[h] * A.ld + ak[h];
    } else {
      afix[h] = m0 + (t % 16) * 4;
      ak[h] = kbeg + t / 16;
      aok[h] = true;
      aoff[h] = (int64_t)ak[h] * A.ld + afix[h];
    }
    if (BROW) {
      bfix[h] = n0 + t / KQ;
      bk[h] = kbeg + (t % KQ) * 4;
      bok[h] = bfix[h] < N;
      boff[h] = bfix[h] * B.ld + bk[h];
    } else {
      bfix[h] = n0 + (t % 16) * 4;
      bk[h] = kbeg + t / 16;
      bok[h] = true;
      boff[h] = (int64_t)bk[h] * B.ld + bfix[h];
    }
  }
  const int64_t astep = AROW ? BK : (int64_t)BK * A.ld;
  const int64_t bstep = BROW ? BK : (int64_t)BK * B.ld;

  float4 ra[H], rb[H];
  auto load = [&](int slab) {
#pragma unroll
    for (int h = 0; h < H; ++h) {
      const int32_t ka = ak[h] + slab * BK;
      const int64_t ao = aoff[h] + slab * astep;
      // k-contiguous: columns are k; row-contiguous: row k, columns afix..afix+3
      ra[h] = AROW ? load4<AV>(A.p, ao, aok[h], ka, kend) : load4<AV>(A.p, ao, ka < kend, afix[h], M);
      const int32_t kb = bk[h] + slab * BK;
      const int64_t bo = boff[h] + slab * bstep;
      rb[h] = BROW ? load4<BV>(B.p, bo, bok[h], kb, kend) : load4<BV>(B.p, bo, kb < kend, bfix[h], N);
    }
  };
  auto store = [&](int buf) {
#pragma unroll
    for (int h = 0; h < H; ++h) {
      const int t = tid + kThreads * h;
      if (AROW) {
        *reinterpret_cast<float4*>(&As[buf][(t / KQ) * KPR + (t % KQ) * 4]) = ra[h];
      } else {
        float* d = &As[buf][(t / 16) * KPC + (t % 16) * 4];
        d[0] = ra[h].x;
        d[1] = ra[h].y;
        d[2] = ra[h].z;
        d[3] = ra[h].w;
      }
      if (BROW) {
        *reinterpret_cast<float4*>(&Bs[buf][(t / KQ) * KPR + (t % KQ) * 4]) = rb[h];
      } else {
        float* d = &Bs[buf][(t / 16) * KPC + (t % 16) * 4];
        d[0] = rb[h].x;
        d[1] = rb[h].y;
        d[2] = rb[h].z;
        d[3] = rb[h].w;
      }
    }
  };
  // operand values of this lane for MFMA step j: rows base + 16 i + c16, k = KQ g + j
  auto fetch = [&](const float* S, bool row_layout, int base, float (&v)[2][KQ]) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      if (row_layout) {
        const float* p = S + (base + 16 * i + c16) * KPR + KQ * g;
#pragma unroll
        for (int q = 0; q < KQ / 4; ++q) {
          const float4 x = *reinterpret_cast<const float4*>(p + 4 * q);
          v[i][4 * q + 0] = x.x;
          v[i][4 * q + 1] = x.y;
          v[i][4 * q + 2] = x.z;
          v[i][4 * q + 3] = x.w;
        }
      } else {
#pragma unroll
        for (int j = 0; j < KQ; ++j) v[i][j] = S[(KQ * g + j) * KPC + base + 16 * i + c16];
      }
    }
  };

  const int nk = (kend - kbeg + BK - 1) / BK;
  load(0);
  store(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) load(kt + 1);
    float av[2][KQ], bv[2][KQ];
    fetch(As[buf], AROW, wm, av);
    fetch(Bs[buf], BROW, wn, bv);
#pragma unroll
    for (int j = 0; j < KQ; ++j) {
      acc[0][0] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[0][j], bv[0][j], acc[0][0], 0, 0, 0);
      acc[0][1] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[0][j], bv[1][j], acc[0][1], 0, 0, 0);
      acc[1][0] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[1][j], bv[0][j], acc[1][0], 0, 0, 0);
      acc[1][1] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[1][j], bv[1][j], acc[1][1], 0, 0, 0);
    }
    if (kt + 1 < nk) store(buf ^ 1);
    __syncthreads();
  }

  // D layout of 16x16x4: lane l holds rows 4*(l/16) + r, column l%16
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t gm_ = m0 + wm + 16 * i + 4 * g + r;
        const int64_t gn_ = n0 + wn + 16 * j + c16;
        if (gm_ < M && gn_ < N) out_store(C, gm_, gn_, acc[i][j][r], epilogue);
      }
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

}  // namespace

int launch_gemm(const MatView& A, const MatView& B, const OutView& C, int32_t m_cap, int32_t N,
                int32_t k_cap, const int32_t* m_dev, const int32_t* k_dev, int32_t epilogue,
                int32_t split_min_chunk, hipStream_t st) {
  if (m_cap <= 0 || N <= 0 || k_cap <= 0) return GNN_OK;
  if (!A.p || !B.p || !C.p0) return fail(GNN_EINVAL, "gemm: null operand");
  if (A.trans && B.trans) return fail(GNN_EINVAL, "gemm: both operands transposed");
  const int64_t gm = ceil_div(m_cap, BM), gn = ceil_div(N, BN);
  const int64_t gm8 = ceil_div(gm, kXcds) * kXcds;  // m-tiles rounded up to whole XCD rounds
  int64_t gz = 1;
  const int32_t min_chunk = split_min_chunk > BK ? split_min_chunk : BK;
  if (epilogue == 2 && split_min_chunk > 0) {
    // enough splits to fill the GPU at the capacity; the kernel trims them to
    // the live reduction length
    const int64_t want = std::max<int64_t>(1, 1024 / (gm * gn));
    gz = std::min<int64_t>(want, std::max<int64_t>(1, ceil_div(k_cap, min_chunk)));
  }
  if (gm8 * gn > INT32_MAX / 2 || gz > 65535) return fail(GNN_EINVAL, "gemm: grid too large");
  Out o{C.p0, C.p1 ? C.p1 : C.p0, C.ld0, C.p1 ? C.ld1 : C.ld0, C.split, C.axis};
  Operand a{A.p, A.ld, 0};
  Operand b{B.p, B.ld, 0};
  // vector loads: 16-byte aligned rows, and the extent of the contiguous axis
  // a multiple of 4
  a.vec = aligned16(A.p) && A.ld % 4 == 0 && (A.trans ? m_cap % 4 == 0 : k_cap % 4 == 0);
  b.vec = aligned16(B.p) && B.ld % 4 == 0 && (B.trans ? k_cap % 4 == 0 : N % 4 == 0);
  const int code = (A.trans ? 8 : 0) | (B.trans ? 4 : 0) | (a.vec ? 2 : 0) | (b.vec ? 1 : 0);
  const dim3 grid((unsigned)(gm8 * gn), 1, (unsigned)gz);
#define GNN_GEMM_CASE(AT, BT, AV, BV)                                                        \
  case (AT * 8 + BT * 4 + AV * 2 + BV):                                                      \
    gemm_kernel<AT, BT, AV, BV><<<grid, kThreads, 0, st>>>(a, b, o, m_cap, N, k_cap, m_dev, \
                                                           k_dev, epilogue, min_chunk);      \
    break;
#define GNN_GEMM_CASES_AB(AT, BT) \
  GNN_GEMM_CASE(AT, BT, 0, 0)     \
  GNN_GEMM_CASE(AT, BT, 0, 1)     \
  GNN_GEMM_CASE(AT, BT, 1, 0)     \
  GNN_GEMM_CASE(AT, BT, 1, 1)
  switch (code) {
    GNN_GEMM_CASES_AB(0, 0)
    GNN_GEMM_CASES_AB(1, 0)
    GNN_GEMM_CASES_AB(0, 1)
    default: return fail(GNN_EINVAL, "gemm: unsupported operand combination");
  }
#undef GNN_GEMM_CASES_AB
#undef GNN_GEMM_CASE
  GNN_LAUNCH_CHECK("gemm");
  return GNN_OK;
}

}  // namespace gnn
