"""GPU feature caching of a host-resident feature table (CPU oracle).

Part of the CPU oracle (test infrastructure).

What the paper fixes (section 3, GPU Feature Caching): the feature table stays
in host memory, a set of frequently accessed rows is kept in GPU memory, and
a fetch serves a row from GPU memory when it is there and over the host link
otherwise; the rows kept are chosen by least-recently-used replacement (the
approach of HugeCTR's GPU embedding cache, which the paper integrates).
Readings taken where the paper is silent:

* organisation: num_sets sets of `ways` entries (set-associative, like
  HugeCTR's cache); node v belongs to set fmix32(v) mod num_sets, fmix32 being
  the 32-bit finaliser of MurmurHash3 (Appleby);
* recency is counted in fetch calls (batches): call t (1, 2, ...) stamps
  every entry it reads with t;
* after the lookups of a call, each set takes in its missed nodes, in order
  of their position in the request, as long as it has entries not read by
  this call; those entries are replaced oldest stamp first (never-used
  entries, stamp 0, first; ties: lower way).  Missed nodes beyond that are
  served from host memory without being cached;
* the requested ids of one call are distinct (a block's node list is).
"""
from __future__ import annotations

import numpy as np

MASK32 = 0xFFFFFFFF


def fmix32(h: int) -> int:
    """MurmurHash3's 32-bit finaliser (a bijection of 32-bit words)."""
    h &= MASK32
    h ^= h >> 16
    h = (h * 0x85EBCA6B) & MASK32
    h ^= h >> 13
    h = (h * 0xC2B2AE35) & MASK32
    h ^= h >> 16
    return h


def set_of(v: int, num_sets: int) -> int:
    return fmix32(v) % num_sets


class FeatureCache:
    """State: key[s][w] (-1 = empty), stamp[s][w] (0 = never used), the cached
    row of every entry, and the number of calls so far."""

    def __init__(self, num_sets: int, ways: int, width: int, dtype=np.float32):
        assert num_sets >= 1 and 1 <= ways <= 64 and width >= 1
        self.S, self.W, self.F = num_sets, ways, width
        self.key = np.full((num_sets, ways), -1, dtype=np.int64)
        self.stamp = np.zeros((num_sets, ways), dtype=np.int64)
        self.rows = np.zeros((num_sets, ways, width), dtype=dtype)
        self.calls = 0

    def fetch(self, X: np.ndarray, ids):
        """Rows X[ids] (served from the cache where possible), then the
        replacement step.  Returns (rows, hits, misses)."""
        ids = [int(v) for v in ids]
        assert len(set(ids)) == len(ids), "requested ids must be distinct"
        self.calls += 1
        t = self.calls
        out = np.zeros((len(ids), self.F), dtype=self.rows.dtype)
        missed = {}  # set -> request positions, in request order
        hits = 0
        for i, v in enumerate(ids):
            s = set_of(v, self.S)
            way = [w for w in range(self.W) if self.key[s, w] == v]
            if way:
                w = way[0]
                out[i] = self.rows[s, w]
                self.stamp[s, w] = t
                hits += 1
            else:
                out[i] = X[v]
                missed.setdefault(s, []).append(i)
        for s, positions in missed.items():
            victims = sorted((w for w in range(self.W) if self.stamp[s, w] < t),
                             key=lambda w: (self.stamp[s, w], w))
            for i, w in zip(positions, victims):
                self.key[s, w] = ids[i]
                self.stamp[s, w] = t
                self.rows[s, w] = X[ids[i]]
        return out, hits, len(ids) - hits

    def contents(self):
        """{node id: (set, way, stamp)} of the cached rows."""
        out = {}
        for s in range(self.S):
            for w in range(self.W):
                if self.key[s, w] >= 0:
                    out[int(self.key[s, w])] = (s, w, int(self.stamp[s, w]))
        return out
