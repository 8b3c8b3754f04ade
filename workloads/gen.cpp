// Host-side synthetic input generator: power-law graphs (R-MAT, Chung-Lu), CSR
// construction, Gaussian feature rows.  Seeded and counter-based, so the result
// does not depend on the number of threads.  It holds none of the training
// method's arithmetic; both the CPU oracle and the GPU library consume what it
// writes.
//
// Build: g++ -O3 -fopenmp -shared -fPIC gen.cpp -o libwlgen.so
#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <omp.h>

namespace {

// SplitMix64 finaliser (Steele, Lea, Flood, "Fast splittable pseudorandom
// number generators", OOPSLA 2014) used as a stateless hash of a counter.
inline uint64_t mix64(uint64_t z) {
  z += 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

inline uint64_t stream_word(uint64_t seed, uint64_t a, uint64_t b) {
  return mix64(mix64(seed ^ mix64(a)) ^ (b * 0xD1B54A32D192ED03ull));
}

// stream_word split in two: the key of (seed, a) once, then one word per b.
inline uint64_t stream_key(uint64_t seed, uint64_t a) { return mix64(seed ^ mix64(a)); }
inline uint64_t keyed_word(uint64_t key, uint64_t b) {
  return mix64(key ^ (b * 0xD1B54A32D192ED03ull));
}

// 53-bit uniform in [0, 1).
inline double u01(uint64_t w) { return (double)(w >> 11) * (1.0 / 9007199254740992.0); }

inline uint16_t f32_to_bf16_rne(float f) {
  uint32_t u;
  std::memcpy(&u, &f, 4);
  if ((u & 0x7F800000u) == 0x7F800000u) return (uint16_t)(u >> 16);  // inf / nan
  uint32_t lsb = (u >> 16) & 1u;
  u += 0x7FFFu + lsb;
  return (uint16_t)(u >> 16);
}

}  // namespace

extern "C" {

// R-MAT (Chakrabarti, Zhan, Faloutsos, SDM 2004): pair i picks one quadrant per
// level with probabilities (a, b, c, 1-a-b-c).  Pairs whose endpoint falls at or
// beyond n are marked with -1 (rejected).
void wl_rmat_pairs(int64_t n_pairs, int32_t scale, int64_t n, double a, double b, double c,
                   uint64_t seed, int32_t* src, int32_t* dst) {
  const double ab = a + b, abc = a + b + c;
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n_pairs; ++i) {
    uint64_t u = 0, v = 0;
    const uint64_t key = stream_key(seed, (uint64_t)i);
    for (int32_t l = 0; l < scale; ++l) {
      double r = u01(keyed_word(key, (uint64_t)l));
      // quadrant a (0, 0), b (0, 1), c (1, 0), d (1, 1), without branches
      const uint64_t ga = r >= a, gab = r >= ab, gabc = r >= abc;
      const uint64_t bu = gab, bv = ga ^ gab ^ gabc;
      u = (u << 1) | bu;
      v = (v << 1) | bv;
    }
    if ((int64_t)u >= n || (int64_t)v >= n) { src[i] = -1; dst[i] = -1; }
    else { src[i] = (int32_t)u; dst[i] = (int32_t)v; }
  }
}

// Chung-Lu: both endpoints of pair i are drawn independently with probability
// proportional to the node weight; cdf[j] = sum_{t<=j} w_t / sum w, cdf[n-1] = 1.
void wl_chunglu_pairs(int64_t n_pairs, const double* cdf, int64_t n, uint64_t seed,
                      int32_t* src, int32_t* dst) {
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n_pairs; ++i) {
    for (int side = 0; side < 2; ++side) {
      double r = u01(stream_word(seed, (uint64_t)i, (uint64_t)side));
      int64_t j = std::upper_bound(cdf, cdf + n, r) - cdf;
      if (j >= n) j = n - 1;
      (side ? dst : src)[i] = (int32_t)j;
    }
  }
}

// Relabel both endpoints through a permutation (skips rejected pairs).
void wl_permute_pairs(int64_t n_pairs, const int32_t* perm, int32_t* src, int32_t* dst) {
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n_pairs; ++i) {
    if (src[i] >= 0) { src[i] = perm[src[i]]; dst[i] = perm[dst[i]]; }
  }
}

// Degree count of the symmetrised multigraph without self loops:
// deg[u] += 1 and deg[v] += 1 for every kept pair (u, v), u != v.
void wl_count_degrees(int64_t n_pairs, const int32_t* src, const int32_t* dst, int64_t* deg) {
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n_pairs; ++i) {
    int32_t u = src[i], v = dst[i];
    if (u < 0 || u == v) continue;
    __atomic_fetch_add(&deg[u], 1, __ATOMIC_RELAXED);
    __atomic_fetch_add(&deg[v], 1, __ATOMIC_RELAXED);
  }
}

// Scatter both directions into rows; cursor starts as a copy of the row offsets.
void wl_scatter_pairs(int64_t n_pairs, const int32_t* src, const int32_t* dst, int64_t* cursor,
                      int32_t* col) {
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n_pairs; ++i) {
    int32_t u = src[i], v = dst[i];
    if (u < 0 || u == v) continue;
    int64_t pu = __atomic_fetch_add(&cursor[u], 1, __ATOMIC_RELAXED);
    int64_t pv = __atomic_fetch_add(&cursor[v], 1, __ATOMIC_RELAXED);
    col[pu] = v;
    col[pv] = u;
  }
}

// Sort every row ascending and drop duplicates in place; newdeg[r] receives the
// unique count (the unique entries occupy the row's prefix).
void wl_sort_unique_rows(int64_t n, const int64_t* rowptr, int32_t* col, int64_t* newdeg) {
#pragma omp parallel for schedule(dynamic, 1024)
  for (int64_t r = 0; r < n; ++r) {
    int32_t* b = col + rowptr[r];
    int32_t* e = col + rowptr[r + 1];
    std::sort(b, e);
    newdeg[r] = std::unique(b, e) - b;
  }
}

// Copy the unique prefix of every row into the compact CSR.
void wl_compact_rows(int64_t n, const int64_t* old_rowptr, const int32_t* old_col,
                     const int64_t* rowptr, int32_t* col) {
#pragma omp parallel for schedule(dynamic, 1024)
  for (int64_t r = 0; r < n; ++r) {
    std::memcpy(col + rowptr[r], old_col + old_rowptr[r],
                (size_t)(rowptr[r + 1] - rowptr[r]) * sizeof(int32_t));
  }
}

// Standard-normal feature rows [row_lo, row_hi) x f, written at out with the
// given row stride (elements).  Element (r, j) depends only on (seed, r, j):
// Box-Muller on the pair of uniforms keyed by (r, j/2).
void wl_normal_rows_f32(int64_t row_lo, int64_t row_hi, int32_t f, int64_t stride, uint64_t seed,
                        float* out) {
#pragma omp parallel for schedule(static)
  for (int64_t r = row_lo; r < row_hi; ++r) {
    float* o = out + (r - row_lo) * stride;
    const uint64_t key = stream_key(seed, (uint64_t)r);
    for (int32_t j = 0; j < f; j += 2) {
      uint64_t w0 = keyed_word(key, (uint64_t)j);
      uint64_t w1 = keyed_word(key, (uint64_t)j + 1);
      double u1 = 1.0 - u01(w0);  // (0, 1]
      double u2 = u01(w1);
      double rad = std::sqrt(-2.0 * std::log(u1));
      o[j] = (float)(rad * std::cos(6.283185307179586 * u2));
      if (j + 1 < f) o[j + 1] = (float)(rad * std::sin(6.283185307179586 * u2));
    }
  }
}

void wl_normal_rows_bf16(int64_t row_lo, int64_t row_hi, int32_t f, int64_t stride, uint64_t seed,
                         uint16_t* out) {
#pragma omp parallel for schedule(static)
  for (int64_t r = row_lo; r < row_hi; ++r) {
    uint16_t* o = out + (r - row_lo) * stride;
    const uint64_t key = stream_key(seed, (uint64_t)r);
    for (int32_t j = 0; j < f; j += 2) {
      uint64_t w0 = keyed_word(key, (uint64_t)j);
      uint64_t w1 = keyed_word(key, (uint64_t)j + 1);
      double u1 = 1.0 - u01(w0);
      double u2 = u01(w1);
      double rad = std::sqrt(-2.0 * std::log(u1));
      o[j] = f32_to_bf16_rne((float)(rad * std::cos(6.283185307179586 * u2)));
      if (j + 1 < f) o[j + 1] = f32_to_bf16_rne((float)(rad * std::sin(6.283185307179586 * u2)));
    }
  }
}

int32_t wl_num_threads(void) { return omp_get_max_threads(); }

}  // extern "C"
