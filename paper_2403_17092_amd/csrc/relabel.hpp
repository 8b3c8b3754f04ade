// The relabelling state of the neighbour sampler shared with the launch that
// finishes a sampling call (the last hop's edge compaction can run inside the
// next launch of a training step, the feature gather).
#pragma once
#include <hip/hip_runtime.h>

#include <cstdint>

namespace gnn {

// Persistent header of the sampler's workspace: a magic word, the last
// finished epoch, this call's top epoch and the node count the per-node words
// were built for.
constexpr uint32_t kMagic = 0x474E4E53u;  // "GNNS"

struct Header {
  uint32_t magic;
  uint32_t done_epoch;
  uint32_t top_epoch;
  uint32_t pad;
  int64_t num_nodes;
};

// Edge compaction of one hop: padded slot (i, r), r < k_i, becomes
// indices[indptr[i] + r] = local id of its key, and adds 1 to src_occ of it.
struct IndexJob {
  const int32_t* nbr_pad;  // [n_dst x fanout], -1 = unused
  const int32_t* kcount;   // [n_dst]
  const int32_t* indptr;
  const int32_t* counts;   // counts[0] = n_dst
  const int32_t* nid;      // per-node local id of this hop
  int32_t* indices;
  int32_t* src_occ;
  int32_t fanout;
  int32_t cap_src;
  int64_t num_nodes;
};

__device__ __forceinline__ void index_slots(const IndexJob& j, int64_t first, int64_t stride) {
  // Four slots per pass, their independent loads (count, pick, row start)
  // issued together and then the four id lookups, so a thread waits on two
  // memory round trips per pass rather than three per slot.
  constexpr int kBatch = 4;
  const int64_t slots = (int64_t)j.counts[0] * j.fanout;
  for (int64_t base = first; base < slots; base += kBatch * stride) {
    int64_t i[kBatch];
    int32_t r[kBatch], kc[kBatch], key[kBatch], at[kBatch], id[kBatch];
#pragma unroll
    for (int k = 0; k < kBatch; ++k) {
      const int64_t s = base + k * stride;
      const bool live = s < slots;
      i[k] = live ? s / j.fanout : 0;
      r[k] = live ? (int32_t)(s - i[k] * j.fanout) : 0;  // dead slots: r = kc = 0, skipped
      kc[k] = live ? j.kcount[i[k]] : 0;
      key[k] = live ? j.nbr_pad[s] : -1;
      at[k] = live ? j.indptr[i[k]] : 0;
    }
#pragma unroll
    for (int k = 0; k < kBatch; ++k) {
      // a pick dropped as an invalid id (device error raised) points at row 0
      const bool ok = r[k] < kc[k] && key[k] >= 0 && (int64_t)key[k] < j.num_nodes;
      id[k] = ok ? j.nid[key[k]] : 0;
    }
#pragma unroll
    for (int k = 0; k < kBatch; ++k) {
      if (r[k] >= kc[k]) continue;
      j.indices[at[k] + r[k]] = id[k];
      const bool ok = key[k] >= 0 && (int64_t)key[k] < j.num_nodes;
      if (ok && (uint32_t)id[k] < (uint32_t)j.cap_src) atomicAdd(&j.src_occ[id[k]], 1);
    }
  }
}

// The transpose of a compacted block (per src node u, the dst nodes v of its
// edges), for the backward of the aggregation as a gather.  Built in two
// steps riding on later sampling launches: an exclusive scan of the
// per-src edge counts (src_occ less the dst's own 1) into t_ptr and the
// cursors t_cur, then a fill that appends every edge's v to its u's list
// (list order unspecified).
struct TransposeJob {
  const int32_t* indptr;
  const int32_t* indices;
  const int32_t* counts;   // counts[0] = n_dst, counts[1] = n_src
  const int32_t* src_occ;
  int32_t* t_ptr;          // [cap_src + 1]
  int32_t* t_cur;          // [cap_src]
  int32_t* t_dst;          // [cap_edges]
  int32_t fanout;
  int32_t cap_src;
};

__device__ __forceinline__ void transpose_fill(const TransposeJob& t, int64_t first, int64_t stride) {
  if (!t.t_dst) return;
  const int64_t slots = (int64_t)t.counts[0] * t.fanout;
  for (int64_t s = first; s < slots; s += stride) {
    const int32_t v = (int32_t)(s / t.fanout);
    const int32_t r = (int32_t)(s - (int64_t)v * t.fanout);
    const int32_t e0 = t.indptr[v];
    if (r >= t.indptr[v + 1] - e0) continue;
    const int32_t u = t.indices[e0 + r];
    if ((uint32_t)u >= (uint32_t)t.cap_src) continue;
    const int32_t pos = atomicAdd(&t.t_cur[u], 1);
    // (a list only overflows with a device error raised: an invalid pick
    // counted nowhere but pointing at row 0)
    if (pos < t.t_ptr[u + 1]) t.t_dst[pos] = v;
  }
}

// Calls that may follow one another without a begin launch ("chained":
// the previous call's last step has already prepared the next one); the
// epoch check of the begin launch keeps room for that many.
constexpr uint32_t kChainCalls = 1024;

// The last step of a sampling call: the last hop's compaction, the fill of a
// pending transpose, and (by the first thread) the header marking the
// per-node words as built for this node count up to this call's epochs.  It
// also prepares a chained next call: the per-call scan state is cleared and
// the next call's epochs are reserved (a begin launch sets them again).
struct SampleTail {
  IndexJob job;
  Header* hdr;
  TransposeJob tfill;
  int32_t* zero;  // the per-call scan state
  int64_t n_zero;
  uint32_t L;
};

__device__ __forceinline__ void finish_sampling(const SampleTail& t, int64_t block, int64_t blocks,
                                                int threads) {
  index_slots(t.job, block * threads + threadIdx.x, blocks * threads);
  transpose_fill(t.tfill, block * threads + threadIdx.x, blocks * threads);
  for (int64_t i = block * threads + threadIdx.x; i < t.n_zero; i += blocks * threads) t.zero[i] = 0;
  if (block == 0 && threadIdx.x == 0) {
    const uint32_t top = t.hdr->top_epoch;
    t.hdr->done_epoch = top;
    t.hdr->top_epoch = top + t.L;
    t.hdr->num_nodes = t.job.num_nodes;
    t.hdr->magic = kMagic;
  }
}

}  // namespace gnn
