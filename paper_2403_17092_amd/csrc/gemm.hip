// Dense update GEMMs of a layer (the transformation step, paper section 2.1):
// forward Z = X W with X = [H_dst | agg] (GraphSAGE) or agg (GCN) and W the
// stacked layer weights, backward dW = X^T dZ (split over rows, atomically
// reduced) and dX = dZ W^T.
//
// Tiling for CDNA4: 64 x 64 x 32 block tiles, 256 threads = four wave64s, each
// owning a 32 x 32 sub-tile computed with v_mfma_f32_16x16x4_f32 (2 x 2 MFMA
// tiles), or, for products on bf16 operands, v_mfma_f32_16x16x32_bf16 (one
// per slab and sub-tile: the operands are staged in fp32 and rounded to bf16
// as they are fed to the matrix cores).  Products with few output tiles take
// 64 x 32 tiles (32 x 16 per wave, 2 x 1 MFMA tiles) so that most CUs hold
// several independent tiles; the accumulation order is the same.  Operands
// are staged through double-buffered LDS fed from two
// register sets, so the global loads of slab k + 2 are in flight while slab k
// feeds the matrix cores; one barrier per slab suffices.  Global loads are 128-bit along each operand's
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
constexpr int kCusPerXcd = 32;
constexpr int kFillBlocks = 256;     // split-K: blocks wanted however short the reduction
constexpr int kMaxSplitBlocks = 1024;
// fp32 products with at most this many 64-wide output tiles at the capacity
// run 32-wide tiles (a split weight gradient only over at most kNarrowRows
// rows: over more, the A tiles read by twice as many blocks cost more than the
// extra blocks gain)
constexpr int64_t kNarrowTiles = 1024;
constexpr int64_t kNarrowRows = 32768;
constexpr int HA = BM * BK / (4 * kThreads);  // staged 4-vectors of A per thread per slab
constexpr int KQ = BK / 4;   // 4-vectors along k in one row of a slab

typedef float floatx4 __attribute__((ext_vector_type(4)));

struct Operand {
  const void* p;      // fp32, or bf16 for an instance with kAH / kBH
  const float* mask;  // ReLU mask of the same layout, or null
  int64_t ld;
  int64_t extent;  // elements from p to one past the operand's last element
  int32_t vec;     // 4-element vector loads allowed (16 bytes; 8 for bf16)
};

// Rows the launch zeroes besides the product (see OutView).
struct ZeroJob {
  float4* p;
  int64_t ld4;
  int32_t c4;
  const int32_t* lo;
  const int32_t* hi;
  int32_t cap;
};

// Flags of a kernel instance: operand transposed, vector loads, masked,
// bf16 products, operand stored as bf16 (read 4 elements = 8 bytes at a time
// and widened exactly; needs vector loads).
enum : int { kAT = 8, kBT = 4, kAV = 2, kBV = 1, kAM = 16, kBM = 32, kBF = 64, kAH = 128, kBH = 256 };

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

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

// Four consecutive outputs (i, j .. j+3), j a multiple of 4; columns at or
// past n_lim are dropped.  A 16-byte store when the row piece is whole, lies
// in one part and is aligned; element stores otherwise.
__device__ __forceinline__ void out_store4(const Out& o, int64_t i, int64_t j, float4 v,
                                           int64_t n_lim) {
  const bool second = o.axis == 0 ? (i >= o.split) : (j >= o.split);
  const bool one_part = o.axis == 0 || second || j + 3 < o.split;
  int64_t ii = i, jj = j;
  if (second) {
    if (o.axis == 0) ii -= o.split;
    else jj -= o.split;
  }
  float* p = (second ? o.p1 : o.p0) + ii * (second ? o.ld1 : o.ld0) + jj;
  if (one_part && j + 3 < n_lim && (reinterpret_cast<uintptr_t>(p) & 15) == 0) {
    *reinterpret_cast<float4*>(p) = v;
    return;
  }
  const float e[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int t = 0; t < 4; ++t)
    if (j + t < n_lim) out_store(o, i, j + t, e[t], 0);
}

// Operand loads go through buffer resources: an offset past the resource's
// range reads as 0, so a masked element costs no branch and the compiler can
// count the loads in flight exactly.
constexpr int32_t kBufWord3 = 0x00020000;  // raw untyped buffer (gfx9 family)
constexpr uint32_t kOob = 0x80000000u;     // beyond every range below

// Resource over element o on of an operand of ES-byte elements (clamped to
// 2^31 - 1 bytes of the operand's extent).
template <int ES>
__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc_from(const void* base, int64_t extent,
                                                            int64_t o) {
  int64_t bytes = (extent - o) * ES;
  bytes = bytes < 0 ? 0 : (bytes > 0x7FFFFFFF ? 0x7FFFFFFF : bytes);
  char* p = const_cast<char*>(static_cast<const char*>(base)) + o * ES;
  return __builtin_amdgcn_make_buffer_rsrc(p, (short)0, (int)bytes, kBufWord3);
}

__device__ __forceinline__ float4 relu_masked(float4 x, float4 m) {
  return make_float4(m.x > 0.f ? x.x : 0.f, m.y > 0.f ? x.y : 0.f, m.z > 0.f ? x.z : 0.f,
                     m.w > 0.f ? x.w : 0.f);
}

// Four consecutive elements at byte offset `off` of resource r; element e
// reads 0 unless `valid` and c + e < c_lim.  VEC needs c and c_lim to be
// multiples of 4, so a chunk is entirely valid or not.
template <bool VEC, bool HALF = false>
__device__ __forceinline__ float4 load4(__amdgpu_buffer_rsrc_t r, uint32_t off, bool valid,
                                        int64_t c, int64_t c_lim) {
  if constexpr (HALF) {
    // four bf16 (8 bytes), widened exactly
    static_assert(VEC, "bf16 operands are read as vectors");
    const uint32_t o = (valid && c < c_lim) ? off : kOob;
    const auto x = __builtin_amdgcn_raw_buffer_load_b64(r, o, 0, 0);
    const uint32_t w0 = (uint32_t)x[0], w1 = (uint32_t)x[1];
    return make_float4(__uint_as_float(w0 << 16), __uint_as_float(w0 & 0xFFFF0000u),
                       __uint_as_float(w1 << 16), __uint_as_float(w1 & 0xFFFF0000u));
  }
  if (VEC) {
    const uint32_t o = (valid && c < c_lim) ? off : kOob;
    const auto x = __builtin_amdgcn_raw_buffer_load_b128(r, o, 0, 0);
    return make_float4(__uint_as_float(x[0]), __uint_as_float(x[1]), __uint_as_float(x[2]),
                       __uint_as_float(x[3]));
  }
  float v[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const uint32_t o = (valid && (c + e) < c_lim) ? off + 4 * e : kOob;
    v[e] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, o, 0, 0));
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
// Blocks past gemm_blocks zero the ZeroJob's rows instead.
struct GemmArgs {
  Operand A, B;
  Out C;
  int32_t m_cap, N, k_cap;
  const int32_t* m_dev;
  const int32_t* k_dev;
  int32_t epilogue, min_chunk, nsplit, gemm_blocks;
  ZeroJob zj;
  FillPair fills;
};

// LDS floats of an instance with TN-column tiles: two stages of both
// operands, or the output tile
template <int FL, int TN>
constexpr int gemm_smem() {
  constexpr bool AROW = !(FL & kAT), BROW = FL & kBT;
  constexpr int AE = AROW ? BM * (BK + 4) : BK * (BM + 1);
  constexpr int BE = BROW ? TN * (BK + 4) : BK * (TN + 1);
  constexpr int T = BM * (TN + 4);
  return 2 * (AE + BE) > T ? 2 * (AE + BE) : T;
}

// One GEMM launch's work for block `bid` of `nbid` (its grid part), with the
// LDS at smem (gemm_smem<FL, TN>() floats): output tiles of BM rows and TN
// columns (64, or 32 where 64-wide tiles would leave most CUs one tile).
template <int FL, int TN>
__device__ __forceinline__ void gemm_body(const GemmArgs& ga, int32_t bid, int32_t nbid, float* smem) {
  const Operand A = ga.A, B = ga.B;
  const Out C = ga.C;
  const int32_t m_cap = ga.m_cap, N = ga.N, k_cap = ga.k_cap;
  const int32_t* m_dev = ga.m_dev;
  const int32_t* k_dev = ga.k_dev;
  const int32_t epilogue = ga.epilogue, min_chunk = ga.min_chunk, nsplit = ga.nsplit;
  const int32_t gemm_blocks = ga.gemm_blocks;
  const ZeroJob zj = ga.zj;
  constexpr bool AT = FL & kAT, BT = FL & kBT, AV = FL & kAV, BV = FL & kBV;
  constexpr bool AM = FL & kAM, BM_ = FL & kBM, BF = FL & kBF, AH = FL & kAH, BH = FL & kBH;
  constexpr int AES = AH ? 2 : 4, BES = BH ? 2 : 4;  // element bytes
  static_assert(!(AM && AH) && !(BM_ && BH), "masks go with fp32 operands");
  if (bid >= gemm_blocks) {
    if (zj.p) {
      const int32_t lo = zj.lo ? *zj.lo : 0;
      int32_t hi = *zj.hi;
      hi = hi > zj.cap ? zj.cap : hi;
      const int64_t n = lo < hi ? (int64_t)(hi - lo) * zj.c4 : 0;
      const int64_t stride = (int64_t)(nbid - gemm_blocks) * kThreads;
      for (int64_t i = (int64_t)(bid - gemm_blocks) * kThreads + threadIdx.x; i < n; i += stride) {
        const int64_t r = lo + i / zj.c4, c = i % zj.c4;
        zj.p[r * zj.ld4 + c] = make_float4(0.f, 0.f, 0.f, 0.f);
      }
    }
    run_fills(ga.fills, bid - gemm_blocks, nbid - gemm_blocks, kThreads);
    return;
  }
  constexpr bool AROW = !AT, BROW = BT;   // [row][k] layouts
  constexpr int KPR = BK + 4;             // row-layout stride
  constexpr int KPCA = BM + 1, KPCB = TN + 1;  // column-layout strides
  constexpr int AE = AROW ? BM * KPR : BK * KPCA;
  constexpr int BE = BROW ? TN * KPR : BK * KPCB;
  constexpr int HB = TN * BK / (4 * kThreads);  // staged 4-vectors of B per thread per slab
  constexpr int WNW = TN / 2;                  // columns of a wave's sub-tile (its rows: 32)
  constexpr int NJ = WNW / 16;                 // 16-column MFMA tiles per wave
  static_assert(HA >= 1 && HB >= 1 && NJ >= 1, "tile sizes");
  // operand staging; after the last slab the same memory holds the output
  // tile for the coalesced store
  constexpr int TS = TN + 4;  // output tile row stride (conflict-free D-layout writes)
  static_assert(2 * (AE + BE) <= gemm_smem<FL, TN>() && BM * TS <= gemm_smem<FL, TN>(), "LDS size");
  float (*As)[AE] = reinterpret_cast<float (*)[AE]>(smem);
  float (*Bs)[BE] = reinterpret_cast<float (*)[BE]>(smem + 2 * AE);

  int32_t M = m_cap, K = k_cap;
  if (m_dev) M = min(M, *m_dev);
  if (k_dev) K = min(K, *k_dev);

  // XCD-aware block order: consecutive block ids go to consecutive XCDs.
  // Without split-K, m-tile mt is owned by XCD mt % 8 and its n-tiles are
  // consecutive blocks of that XCD (they share the A tile in that XCD's L2);
  // live rows below the capacity still spread over all XCDs.  With split-K,
  // split z is owned by XCD z % 8 and its tiles are consecutive blocks there
  // (they share the k-chunk of both operands), so every XCD works even when
  // the output has fewer than eight m-tiles.
  const int gm = (m_cap + BM - 1) / BM, gn = (N + TN - 1) / TN;
  const int b = bid;
  const int xcd = b % kXcds, idx = b / kXcds;
  int64_t mt, nt;
  int32_t z = 0;
  if (nsplit > 1) {
    const int tiles = gm * gn;
    z = (idx / tiles) * kXcds + xcd;
    mt = (idx % tiles) / gn;
    nt = (idx % tiles) % gn;
  } else {
    mt = (int64_t)(idx / gn) * kXcds + xcd;
    nt = idx % gn;
  }
  const int64_t m0 = mt * BM;
  const int64_t n0 = nt * TN;
  if (m0 >= M) return;

  // split-K over the live reduction length
  int32_t kbeg = 0, kend = K;
  if (nsplit > 1) {
    // chunks of at least min_chunk, but enough of them for about one block
    // per CU when the reduction is short
    int32_t parts = (K + min_chunk - 1) / min_chunk;
    const int32_t fill = min((kFillBlocks + gm * gn - 1) / (gm * gn), (K + BK - 1) / BK);
    parts = parts < fill ? fill : parts;
    parts = parts < 1 ? 1 : (parts > nsplit ? nsplit : parts);
    // Split z runs on XCD z % 8, whose CUs share its splits' tiles: a count
    // just past a multiple of 8 gives some XCDs an extra round.  Estimate the
    // time as CU rounds on the busiest XCD times slabs per chunk and keep the
    // count or its round-down to a multiple of 8, whichever is cheaper (the
    // round-down on a tie: fewer partial sums).
    if (parts > kXcds) {
      const int32_t slabs = (K + BK - 1) / BK;
      auto cost = [&](int32_t p) {
        const int32_t per_xcd = (p + kXcds - 1) / kXcds * gm * gn;
        return (per_xcd + kCusPerXcd - 1) / kCusPerXcd * ((slabs + p - 1) / p);
      };
      const int32_t down = parts - parts % kXcds;
      if (cost(down) <= cost(parts)) parts = down;
    }
    if (z >= parts) return;
    int32_t chunk = (K + parts - 1) / parts;
    chunk = (chunk + BK - 1) / BK * BK;
    kbeg = z * chunk;
    kend = min(K, kbeg + chunk);
    if (kbeg >= kend) return;
  }

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = (wave >> 1) * 32, wn = (wave & 1) * WNW;
  const int g = lane >> 4, c16 = lane & 15;

  floatx4 acc[2][NJ];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < NJ; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};

  // Staged 4-vector h of each operand: a k-contiguous operand takes (row
  // t / KQ, k (t % KQ) * 4), a row-contiguous one of W columns (k t / (W /
  // 4), column (t % (W / 4)) * 4) of the slab tile.  Per thread: its byte
  // offset from the tile origin, its k coordinate within the slab, the fixed
  // coordinate (row or column) and its validity.
  constexpr int CA = BM / 4, CB = TN / 4;  // 4-vectors across a row-contiguous slab row
  uint32_t arel[HA], brel[HB];
  int32_t ak[HA], bk[HB];
  int64_t afix[HA], bfix[HB];
  bool aok[HA], bok[HB];
#pragma unroll
  for (int h = 0; h < HA; ++h) {
    const int t = tid + kThreads * h;
    if (AROW) {
      afix[h] = m0 + t / KQ;
      ak[h] = (t % KQ) * 4;
      aok[h] = afix[h] < M;
      arel[h] = (uint32_t)(((t / KQ) * A.ld + ak[h]) * AES);
    } else {
      afix[h] = m0 + (t % CA) * 4;
      ak[h] = t / CA;
      aok[h] = true;
      arel[h] = (uint32_t)((ak[h] * A.ld + (t % CA) * 4) * AES);
    }
  }
#pragma unroll
  for (int h = 0; h < HB; ++h) {
    const int t = tid + kThreads * h;
    if (BROW) {
      bfix[h] = n0 + t / KQ;
      bk[h] = (t % KQ) * 4;
      bok[h] = bfix[h] < N;
      brel[h] = (uint32_t)(((t / KQ) * B.ld + bk[h]) * BES);
    } else {
      bfix[h] = n0 + (t % CB) * 4;
      bk[h] = t / CB;
      bok[h] = true;
      brel[h] = (uint32_t)((bk[h] * B.ld + (t % CB) * 4) * BES);
    }
  }

  // Two register sets: slab s is staged in set s & 1, so the loads of slab
  // kt + 2 are in flight while slab kt feeds the matrix cores.
  constexpr int HM = HA > HB ? HA : HB;
  float4 ra[2][HA], rb[2][HB];
  auto load = [&](int slab, float4 (&la)[HA], float4 (&lb)[HB]) {
    const int64_t k0 = kbeg + (int64_t)slab * BK;
    const int64_t oa = AROW ? m0 * A.ld + k0 : k0 * A.ld + m0;
    const int64_t ob = BROW ? n0 * B.ld + k0 : k0 * B.ld + n0;
    const __amdgpu_buffer_rsrc_t rA = rsrc_from<AES>(A.p, A.extent, oa);
    const __amdgpu_buffer_rsrc_t rB = rsrc_from<BES>(B.p, B.extent, ob);
    __amdgpu_buffer_rsrc_t rAm = rA, rBm = rB;
    if (AM) rAm = rsrc_from<4>(A.mask, A.extent, oa);
    if (BM_) rBm = rsrc_from<4>(B.mask, B.extent, ob);
#pragma unroll
    for (int h = 0; h < HM; ++h) {
      // k-contiguous: columns are k; row-contiguous: row k, columns afix..afix+3
      if (h < HA) {
        const int64_t ka = k0 + ak[h];
        const bool va = AROW ? aok[h] : ka < kend;
        const int64_t ca = AROW ? ka : afix[h], la_lim = AROW ? (int64_t)kend : (int64_t)M;
        la[h] = load4<AV, AH>(rA, arel[h], va, ca, la_lim);
        if (AM) la[h] = relu_masked(la[h], load4<AV>(rAm, arel[h], va, ca, la_lim));
      }
      if (h < HB) {
        const int64_t kb = k0 + bk[h];
        const bool vb = BROW ? bok[h] : kb < kend;
        const int64_t cb = BROW ? kb : bfix[h], lb_lim = BROW ? (int64_t)kend : (int64_t)N;
        lb[h] = load4<BV, BH>(rB, brel[h], vb, cb, lb_lim);
        if (BM_) lb[h] = relu_masked(lb[h], load4<BV>(rBm, brel[h], vb, cb, lb_lim));
      }
    }
  };
  auto store = [&](int buf, const float4 (&la)[HA], const float4 (&lb)[HB]) {
#pragma unroll
    for (int h = 0; h < HM; ++h) {
      const int t = tid + kThreads * h;
      if (h < HA) {
        if (AROW) {
          *reinterpret_cast<float4*>(&As[buf][(t / KQ) * KPR + (t % KQ) * 4]) = la[h];
        } else {
          float* d = &As[buf][(t / CA) * KPCA + (t % CA) * 4];
          d[0] = la[h].x;
          d[1] = la[h].y;
          d[2] = la[h].z;
          d[3] = la[h].w;
        }
      }
      if (h < HB) {
        if (BROW) {
          *reinterpret_cast<float4*>(&Bs[buf][(t / KQ) * KPR + (t % KQ) * 4]) = lb[h];
        } else {
          float* d = &Bs[buf][(t / CB) * KPCB + (t % CB) * 4];
          d[0] = lb[h].x;
          d[1] = lb[h].y;
          d[2] = lb[h].z;
          d[3] = lb[h].w;
        }
      }
    }
  };
  // operand values of this lane for MFMA step j: rows base + 16 i + c16, k =
  // KQ g + j (column layout: stride kpc)
  auto fetch = [&](const float* S, bool row_layout, int kpc, int base, auto& v) {
    constexpr int NI = sizeof(v) / sizeof(v[0]);
#pragma unroll
    for (int i = 0; i < NI; ++i) {
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
        for (int j = 0; j < KQ; ++j) v[i][j] = S[(KQ * g + j) * kpc + base + 16 * i + c16];
      }
    }
  };

  const int nk = (kend - kbeg + BK - 1) / BK;
  // slab kt: its registers (set `cur`) are free once it sits in LDS, so they
  // take the loads of slab kt + 2; slab kt + 1 (set `nxt`) goes to LDS after
  // the MFMAs of slab kt.  Loads and stores are unconditional (slabs past the
  // end read as 0), which keeps the count of loads in flight static.
  auto step = [&](int kt, float4 (&ca)[HA], float4 (&cb)[HB], const float4 (&na)[HA],
                  const float4 (&nb)[HB]) {
    const int buf = kt & 1;
    load(kt + 2, ca, cb);
    float av[2][KQ], bv[NJ][KQ];
    fetch(As[buf], AROW, KPCA, wm, av);
    fetch(Bs[buf], BROW, KPCB, wn, bv);
    if constexpr (BF) {
      // lane group g holds k = KQ g .. KQ g + 7 of the slab: exactly the eight
      // k values a lane feeds to one 16x16x32 bf16 MFMA (KQ = 8)
      static_assert(KQ == 8, "one bf16 MFMA per slab");
      bf16x8 a8[2], b8[NJ];
#pragma unroll
      for (int j = 0; j < KQ; ++j) {
#pragma unroll
        for (int i = 0; i < 2; ++i) a8[i][j] = (__bf16)av[i][j];  // round to nearest even
#pragma unroll
        for (int i = 0; i < NJ; ++i) b8[i][j] = (__bf16)bv[i][j];
      }
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int jn = 0; jn < NJ; ++jn)
          acc[i][jn] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a8[i], b8[jn], acc[i][jn], 0, 0, 0);
    } else {
#pragma unroll
      for (int j = 0; j < KQ; ++j)
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int jn = 0; jn < NJ; ++jn)
            acc[i][jn] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[i][j], bv[jn][j], acc[i][jn], 0, 0, 0);
    }
    store(buf ^ 1, na, nb);
    __syncthreads();
  };
  load(0, ra[0], rb[0]);
  load(1, ra[1], rb[1]);
  store(0, ra[0], rb[0]);
  __syncthreads();
  int kt = 0;
  for (; kt + 1 < nk; kt += 2) {
    step(kt, ra[0], rb[0], ra[1], rb[1]);
    step(kt + 1, ra[1], rb[1], ra[0], rb[0]);
  }
  if (kt < nk) step(kt, ra[0], rb[0], ra[1], rb[1]);

  // D layout of 16x16x4: lane l holds rows 4*(l/16) + r, column l%16
  if (epilogue == 2) {
    // atomic accumulation straight from the D layout (64-byte row segments)
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < NJ; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int64_t gm_ = m0 + wm + 16 * i + 4 * g + r;
          const int64_t gn_ = n0 + wn + 16 * j + c16;
          if (gm_ < M && gn_ < N) out_store(C, gm_, gn_, acc[i][j][r], epilogue);
        }
    return;
  }
  // plain or ReLU store: the tile goes through LDS so that every thread
  // stores whole 16-byte row pieces
  float* T = smem;  // the last slab's barrier has retired every operand read
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < NJ; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float x = acc[i][j][r];
        T[(wm + 16 * i + 4 * g + r) * TS + wn + 16 * j + c16] = epilogue == 1 ? fmaxf(x, 0.f) : x;
      }
  __syncthreads();
#pragma unroll
  for (int q0 = 0; q0 < BM * TN / 4; q0 += kThreads) {
    const int q = q0 + tid;
    const int row = q / (TN / 4), c4 = q % (TN / 4);
    const int64_t gi = m0 + row, gj = n0 + 4 * c4;
    if (gi >= M || gj >= N) continue;
    const float4 v = *reinterpret_cast<const float4*>(&T[row * TS + 4 * c4]);
    out_store4(C, gi, gj, v, N);
  }
}

template <int FL, int TN>
__global__ void __launch_bounds__(kThreads) gemm_kernel(GemmArgs ga) {
  __shared__ __align__(16) float smem[gemm_smem<FL, TN>()];
  gemm_body<FL, TN>(ga, (int32_t)blockIdx.x, (int32_t)gridDim.x, smem);
}

// Two independent products in one launch (a layer's weight gradient, split
// over rows in 64-wide tiles, and its input gradient in TN2-wide tiles):
// blocks [0, part1) run the first, the others the second.  part1 is a
// multiple of 8, so both keep their XCD-aware block order.
template <int FL1, int FL2, int TN2>
__global__ void __launch_bounds__(kThreads) gemm_pair_kernel(GemmArgs g1, GemmArgs g2, int32_t part1) {
  constexpr int S1 = gemm_smem<FL1, 64>(), S2 = gemm_smem<FL2, TN2>();
  __shared__ __align__(16) float smem[S1 > S2 ? S1 : S2];
  const int32_t b = (int32_t)blockIdx.x;
  if (b < part1) gemm_body<FL1, 64>(g1, b, part1, smem);
  else gemm_body<FL2, TN2>(g2, b - part1, (int32_t)gridDim.x - part1, smem);
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

}  // namespace

namespace {

// A planned launch: the kernel arguments, the instance code and the grid
// (GEMM blocks, then the blocks of the zero job and fills).
struct GemmPlan {
  GemmArgs args;
  int code = 0;
  int tn = 64;         // output tile columns
  int64_t blocks = 0;  // whole grid of this product
  bool empty = false;  // nothing to multiply: only the fills (launch_fill)
};

int plan_gemm(const MatView& A, const MatView& B, const OutView& C, int32_t m_cap, int32_t N,
              int32_t k_cap, const int32_t* m_dev, const int32_t* k_dev, int32_t epilogue,
              int32_t split_min_chunk, GemmPlan* pl, bool allow_narrow = true) {
  if (m_cap <= 0 || N <= 0 || k_cap <= 0) {
    pl->empty = true;
    pl->args.fills = C.fills;
    return GNN_OK;
  }
  if (!C.p0) return fail(GNN_EINVAL, "gemm: null output");
  if (A.trans && B.trans) return fail(GNN_EINVAL, "gemm: both operands transposed");
  const int64_t gm = ceil_div(m_cap, BM);
  int64_t gn = ceil_div(N, BN);
  const int64_t gm8 = ceil_div(gm, kXcds) * kXcds;  // m-tiles rounded up to whole XCD rounds
  const int32_t min_chunk = split_min_chunk > BK ? split_min_chunk : BK;
  const bool split = epilogue == 2 && split_min_chunk > 0;
  // fp32 products with few 64-wide tiles at the capacity take 32-wide
  // tiles: the live rows of a sampled block then give most CUs two or three
  // independent tiles instead of one (forward and dX, split or not; dW, split
  // over rows, unless it runs beside dX in a pair)
  const int shape = (A.trans ? kAT : 0) | (B.trans ? kBT : 0) | (A.mask ? kAM : 0) | (B.mask ? kBM : 0) |
                    (C.bf16 ? kBF : 0) | (A.bf16 ? kAH : 0) | (B.bf16 ? kBH : 0);
  pl->tn = 64;
  const bool narrow_shape = shape == 0 || shape == kBT || shape == (kBT | kAM) ||
                            (split && k_cap <= kNarrowRows && (shape == kAT || shape == (kAT | kBM)));
  if (allow_narrow && gm * gn <= kNarrowTiles && narrow_shape) {
    pl->tn = 32;
    gn = ceil_div(N, 32);
  }
  int64_t gz = 1;
  if (split) {
    // enough splits to fill the GPU at the capacity; the kernel trims them to
    // the live reduction length
    const int64_t want = std::max<int64_t>(1, kMaxSplitBlocks / (gm * gn));
    gz = std::min<int64_t>(want, std::max<int64_t>(1, ceil_div(k_cap, BK)));
  }
  const int64_t blocks = gz > 1 ? ceil_div(gz, kXcds) * kXcds * gm * gn : gm8 * gn;
  if (blocks > INT32_MAX / 4) return fail(GNN_EINVAL, "gemm: grid too large");
  Out o{C.p0, C.p1 ? C.p1 : C.p0, C.ld0, C.p1 ? C.ld1 : C.ld0, C.split, C.axis};
  // physical extents: A is [m x k] (A^T: [k x m]), B is [k x n] (B^T: [n x k])
  const int64_t a_rows = A.trans ? k_cap : m_cap, a_cols = A.trans ? m_cap : k_cap;
  const int64_t b_rows = B.trans ? N : k_cap, b_cols = B.trans ? k_cap : N;
  const void* ap = A.bf16 ? static_cast<const void*>(A.p16) : static_cast<const void*>(A.p);
  const void* bp = B.bf16 ? static_cast<const void*>(B.p16) : static_cast<const void*>(B.p);
  if (!ap || !bp) return fail(GNN_EINVAL, "gemm: null operand");
  Operand a{ap, A.mask, A.ld, (a_rows - 1) * A.ld + a_cols, 0};
  Operand b{bp, B.mask, B.ld, (b_rows - 1) * B.ld + b_cols, 0};
  // tile-relative offsets are 32-bit: 64 rows of the operand must fit
  if (A.ld > (1 << 22) || B.ld > (1 << 22)) return fail(GNN_EINVAL, "gemm: leading dimension too large");
  // vector loads: rows aligned to the vector (16 bytes; 8 for bf16; masks
  // included), and the live extent of the contiguous axis a multiple of 4
  // (so not read from the device)
  auto aligned = [](const void* p, int bytes) {
    return (reinterpret_cast<uintptr_t>(p) & (uintptr_t)(bytes - 1)) == 0;
  };
  a.vec = aligned(ap, A.bf16 ? 8 : 16) && (!A.mask || aligned16(A.mask)) && A.ld % 4 == 0 &&
          (A.trans ? (m_cap % 4 == 0 && !m_dev) : (k_cap % 4 == 0 && !k_dev));
  b.vec = aligned(bp, B.bf16 ? 8 : 16) && (!B.mask || aligned16(B.mask)) && B.ld % 4 == 0 &&
          (B.trans ? (k_cap % 4 == 0 && !k_dev) : N % 4 == 0);
  if ((A.bf16 && (!a.vec || A.mask)) || (B.bf16 && (!b.vec || B.mask)))
    return fail(GNN_EINVAL, "gemm: a bf16 operand needs aligned 4-element rows and no mask");
  if ((A.bf16 || B.bf16) && !C.bf16) return fail(GNN_EINVAL, "gemm: bf16 operands need bf16 products");
  ZeroJob zj{reinterpret_cast<float4*>(C.zero_p), C.zero_ld / 4, C.zero_cols / 4, C.zero_lo,
             C.zero_hi, C.zero_cap};
  int64_t zblocks = 0;
  if (C.zero_p) {
    if (C.zero_ld % 4 || C.zero_cols % 4 || !aligned16(C.zero_p) || !C.zero_hi)
      return fail(GNN_EINVAL, "gemm: zeroed rows must be 16-byte aligned float4 rows");
    zblocks = std::min<int64_t>(1024, std::max<int64_t>(1, ceil_div((int64_t)C.zero_cap * (C.zero_cols / 4),
                                                                      kThreads * 4)));
  }
  pl->code = (A.trans ? kAT : 0) | (B.trans ? kBT : 0) | (a.vec ? kAV : 0) | (b.vec ? kBV : 0) |
             (A.mask ? kAM : 0) | (B.mask ? kBM : 0) | (C.bf16 ? kBF : 0) |
             (A.bf16 ? kAH : 0) | (B.bf16 ? kBH : 0);

  zblocks = std::max<int64_t>(zblocks, fill_blocks(C.fills, kThreads));
  pl->args = GemmArgs{a, b, o, m_cap, N, k_cap, m_dev, k_dev, epilogue, min_chunk, (int32_t)gz,
                      (int32_t)blocks, zj, C.fills};
  pl->blocks = blocks + zblocks;
  return GNN_OK;
}

int launch_empty(const GemmPlan& pl, hipStream_t st) {
  // nothing to multiply; the fills still happen
  FillRange fr[2];
  int n = 0;
  for (int r = 0; r < 2; ++r)
    if (pl.args.fills.n[r] > 0)
      fr[n++] = FillRange{pl.args.fills.p[r], pl.args.fills.n[r], pl.args.fills.v[r]};
  return launch_fill(fr, n, st);
}

int launch_plan(const GemmPlan& pl, const char* name, hipStream_t st) {
  if (pl.empty) return launch_empty(pl, st);
  auto go = [&](auto kernel) { launch(name, kernel, dim3((unsigned)pl.blocks), kThreads, 0, st, pl.args); };
  // instances: forward (A X, B weights), dW (A^T, B = dZ, maybe masked),
  // dX (A = dZ maybe masked, B^T weights); vector and scalar loads each;
  // bf16 products with X stored as bf16: forward, and dW with dZ in fp32
  // (maybe masked) or stored as bf16
#define GNN_GEMM_CASE(F)      \
  case (F):                   \
    go(gemm_kernel<(F), 64>); \
    break;
#define GNN_GEMM_CASES_V(F) GNN_GEMM_CASE(F) GNN_GEMM_CASE(F | kBV) GNN_GEMM_CASE(F | kAV) GNN_GEMM_CASE(F | kAV | kBV)
#define GNN_GEMM_NARROW(F)    \
  case (F):                   \
    go(gemm_kernel<(F), 32>); \
    break;
#define GNN_GEMM_NARROW_V(F) GNN_GEMM_NARROW(F) GNN_GEMM_NARROW(F | kBV) GNN_GEMM_NARROW(F | kAV) GNN_GEMM_NARROW(F | kAV | kBV)
  if (pl.tn == 32) {
    // (the shapes plan_gemm gives 32-wide tiles: forward, dX and split dW in fp32)
    switch (pl.code) {
      GNN_GEMM_NARROW_V(0)
      GNN_GEMM_NARROW_V(kBT)
      GNN_GEMM_NARROW_V(kBT | kAM)
      GNN_GEMM_NARROW_V(kAT)
      GNN_GEMM_NARROW_V(kAT | kBM)
      default: return fail(GNN_EINVAL, "gemm: unsupported operand combination for 32-wide tiles");
    }
    GNN_LAUNCH_CHECK("gemm");
    return GNN_OK;
  }
  switch (pl.code) {
    GNN_GEMM_CASES_V(0)
    GNN_GEMM_CASES_V(kAT)
    GNN_GEMM_CASES_V(kAT | kBM)
    GNN_GEMM_CASES_V(kBT)
    GNN_GEMM_CASES_V(kBT | kAM)
    GNN_GEMM_CASE(kBF | kAH | kAV)
    GNN_GEMM_CASE(kBF | kAH | kAV | kBV)
    GNN_GEMM_CASE(kAT | kBF | kAH | kAV)
    GNN_GEMM_CASE(kAT | kBF | kAH | kAV | kBV)
    GNN_GEMM_CASE(kAT | kBM | kBF | kAH | kAV)
    GNN_GEMM_CASE(kAT | kBM | kBF | kAH | kAV | kBV)
    GNN_GEMM_CASE(kAT | kBF | kAH | kAV | kBH | kBV)
    default: return fail(GNN_EINVAL, "gemm: unsupported operand combination");
  }
#undef GNN_GEMM_NARROW_V
#undef GNN_GEMM_NARROW
#undef GNN_GEMM_CASES_V
#undef GNN_GEMM_CASE
  GNN_LAUNCH_CHECK("gemm");
  return GNN_OK;
}

}  // namespace

int launch_gemm(const MatView& A, const MatView& B, const OutView& C, int32_t m_cap, int32_t N,
                int32_t k_cap, const int32_t* m_dev, const int32_t* k_dev, int32_t epilogue,
                int32_t split_min_chunk, const char* name, hipStream_t st) {
  GemmPlan pl;
  if (int rc = plan_gemm(A, B, C, m_cap, N, k_cap, m_dev, k_dev, epilogue, split_min_chunk, &pl))
    return rc;
  return launch_plan(pl, name, st);
}

int launch_gemm_pair(const GemmSpec& p1, const GemmSpec& p2, const char* name, hipStream_t st) {
  GemmPlan a, b;
  // (the weight gradient of a pair keeps 64-wide tiles)
  if (int rc = plan_gemm(p1.A, p1.B, p1.C, p1.m_cap, p1.N, p1.k_cap, p1.m_dev, p1.k_dev, p1.epilogue,
                         p1.split_min_chunk, &a, false))
    return rc;
  if (int rc = plan_gemm(p2.A, p2.B, p2.C, p2.m_cap, p2.N, p2.k_cap, p2.m_dev, p2.k_dev, p2.epilogue,
                         p2.split_min_chunk, &b))
    return rc;
  // the pairs a hidden layer's backward takes: dW = X^T dZ with dZ masked by
  // the layer's ReLU output or not (the output layer), with dX = dZ W^T the same
  constexpr int kDwM = kAT | kBM | kAV | kBV, kDxM = kBT | kAM | kAV | kBV;
  constexpr int kDw = kAT | kAV | kBV, kDx = kBT | kAV | kBV;
  const bool pair = !a.empty && !b.empty &&
                    ((a.code == kDwM && b.code == kDxM) || (a.code == kDw && b.code == kDx));
  if (!pair) {
    if (int rc = launch_plan(a, p1.name, st)) return rc;
    return launch_plan(b, p2.name, st);
  }
  if (a.tn != 64) return fail(GNN_EINVAL, "gemm pair: the weight gradient takes 64-wide tiles");
  const int64_t part1 = ceil_div(a.blocks, kXcds) * kXcds;  // whole XCD rounds
  if (part1 + b.blocks > INT32_MAX / 2) return fail(GNN_EINVAL, "gemm: grid too large");
  const dim3 grid((unsigned)(part1 + b.blocks));
  auto go = [&](auto kernel) { launch(name, kernel, grid, kThreads, 0, st, a.args, b.args, (int32_t)part1); };
  // (the weight gradient is split over rows, so its tiles are 64 wide)
  if (a.code == kDwM) {
    if (b.tn == 32) go(gemm_pair_kernel<kDwM, kDxM, 32>);
    else go(gemm_pair_kernel<kDwM, kDxM, 64>);
  } else {
    if (b.tn == 32) go(gemm_pair_kernel<kDw, kDx, 32>);
    else go(gemm_pair_kernel<kDw, kDx, 64>);
  }
  GNN_LAUNCH_CHECK("gemm pair");
  return GNN_OK;
}

}  // namespace gnn
