"""Layer-wise uniform neighbour sampling and block construction (CPU oracle).

Part of the CPU oracle (test infrastructure).

What the paper fixes (section 2.2, Neighbor Sampling): every node of the
current frontier gets a random selection of its neighbours, bounded by a
per-layer budget, and an L-layer model samples L hops around each root.  The
readings taken where the paper is silent:

* without replacement; a node with degree <= budget keeps all its neighbours,
  so every node contributes exactly min(budget, degree) edges;
* budgets are given in hop order: fanouts[0] applies to the seeds;
* the k positions are drawn with Floyd's algorithm (Bentley & Floyd, "A sample
  of brilliance", CACM 30(9), 1987) from the Philox stream of (key, hop, node),
  draw s mapped to [0, m) as floor(r_s * m / 2**64); the chosen positions are
  emitted in ascending CSR order, i.e. ascending neighbour id;
* the block of hop h lists its dst nodes (the previous frontier, in order)
  first, followed by every other sampled node in order of first occurrence
  when the edges are scanned by (dst index, position); indices[e] is the local
  id of edge e's neighbour.  The next frontier is that src list.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import List

import numpy as np

from . import philox


def bounded(r: int, m: int) -> int:
    """floor(r * m / 2**64) for a 64-bit draw r: an integer in [0, m)."""
    return (int(r) * int(m)) >> 64


def bounded_vec(r: np.ndarray, m: np.ndarray) -> np.ndarray:
    """Vectorised `bounded` for m < 2**32 (exact)."""
    m = np.asarray(m, dtype=np.uint64)
    assert np.all(m < np.uint64(1 << 32))
    with np.errstate(over="ignore"):
        r = np.asarray(r, dtype=np.uint64)
        rh, rl = r >> np.uint64(32), r & np.uint64(0xFFFFFFFF)
        return ((rh * m + ((rl * m) >> np.uint64(32))) >> np.uint64(32)).astype(np.int64)


def floyd_positions(d: int, k: int, draws) -> List[int]:
    """Floyd's algorithm: a uniform k-subset of {0..d-1}, returned ascending.
    Step s considers j = d-k+s, draws t uniformly from [0, j]; t joins the set
    unless it is already there, in which case j joins instead."""
    chosen: List[int] = []
    for s in range(k):
        j = d - k + s
        t = bounded(draws[s], j + 1)
        chosen.append(j if t in chosen else t)
    return sorted(chosen)


def sample_node(rowptr, col, v: int, fanout: int, rng_key: int, hop: int) -> np.ndarray:
    """Sampled neighbours of node v at hop `hop` (scalar reference)."""
    start, end = int(rowptr[v]), int(rowptr[v + 1])
    d = end - start
    if d <= fanout:
        pos = list(range(d))
    else:
        r = [philox.draw_scalar(rng_key, hop, v, s) for s in range(fanout)]
        pos = floyd_positions(d, fanout, r)
    return np.asarray([col[start + p] for p in pos], dtype=np.int64)


def sample_hop(rowptr, col, dst: np.ndarray, fanout: int, rng_key: int, hop: int):
    """All dst nodes of one hop at once: returns (indptr int64 [n+1], nbr int64 [E]).
    Same steps as `sample_node`, run side by side over the nodes (each node's
    Floyd loop is independent of every other node's)."""
    dst = np.asarray(dst, dtype=np.int64)
    rowptr = np.asarray(rowptr)
    n = dst.shape[0]
    start = rowptr[dst].astype(np.int64)
    deg = rowptr[dst + 1].astype(np.int64) - start
    k = np.minimum(deg, fanout)
    indptr = np.zeros(n + 1, dtype=np.int64)
    np.cumsum(k, out=indptr[1:])
    pos = np.full((n, fanout), -1, dtype=np.int64)

    full = deg <= fanout
    if full.any():
        ar = np.arange(fanout, dtype=np.int64)
        pos[full] = np.where(ar[None, :] < deg[full][:, None], ar[None, :], -1)

    big = ~full
    if big.any():
        d = deg[big]
        r = philox.draws(rng_key, hop, dst[big], fanout)
        picks = np.empty((d.shape[0], fanout), dtype=np.int64)
        for s in range(fanout):
            j = d - fanout + s
            t = bounded_vec(r[:, s], j + 1)
            member = (picks[:, :s] == t[:, None]).any(axis=1) if s else np.zeros_like(t, bool)
            picks[:, s] = np.where(member, j, t)
        pos[big] = np.sort(picks, axis=1)

    valid = pos >= 0
    flat_pos = (start[:, None] + np.where(valid, pos, 0))[valid]  # row-major = (dst, p) order
    nbr = np.asarray(col)[flat_pos].astype(np.int64)
    return indptr, nbr


def relabel(dst: np.ndarray, nbr: np.ndarray):
    """First-occurrence relabelling of [dst, nbr]: returns (src_nodes, indices)."""
    dst = np.asarray(dst, dtype=np.int64)
    nbr = np.asarray(nbr, dtype=np.int64)
    cat = np.concatenate([dst, nbr])
    if cat.size == 0:
        return np.zeros(0, np.int64), np.zeros(0, np.int64)
    uniq, first = np.unique(cat, return_index=True)
    order = np.argsort(first, kind="stable")
    src_nodes = uniq[order]
    rank = np.empty_like(order)
    rank[order] = np.arange(order.shape[0])
    indices = rank[np.searchsorted(uniq, nbr)]
    return src_nodes, indices


def relabel_loop(dst, nbr):
    """The same relabelling as a plain dictionary scan (reference for small inputs)."""
    ids = {}
    src = []
    for v in list(dst) + list(nbr):
        v = int(v)
        if v not in ids:
            ids[v] = len(src)
            src.append(v)
    return np.asarray(src, np.int64), np.asarray([ids[int(v)] for v in nbr], np.int64)


@dataclass
class Block:
    """Bipartite block of one hop: dst nodes are src_nodes[:n_dst]."""
    hop: int
    indptr: np.ndarray     # int64 [n_dst + 1]
    indices: np.ndarray    # int64 [E], local src ids
    src_nodes: np.ndarray  # int64 [n_src], global ids
    nbr: np.ndarray        # int64 [E], global ids (= src_nodes[indices])

    @property
    def n_dst(self) -> int:
        return int(self.indptr.shape[0] - 1)

    @property
    def n_src(self) -> int:
        return int(self.src_nodes.shape[0])

    @property
    def n_edges(self) -> int:
        return int(self.indices.shape[0])


def sample_blocks(rowptr, col, seeds, fanouts, rng_key: int) -> List[Block]:
    """Blocks for hops 1..L (hop order).  Hop h uses fanouts[h-1] and Philox
    counter word 2 = h."""
    frontier = np.asarray(seeds, dtype=np.int64)
    assert np.unique(frontier).shape[0] == frontier.shape[0], "seeds must be distinct"
    blocks = []
    for h, f in enumerate(fanouts, start=1):
        indptr, nbr = sample_hop(rowptr, col, frontier, int(f), rng_key, h)
        src_nodes, indices = relabel(frontier, nbr)
        blocks.append(Block(h, indptr, indices, src_nodes, nbr))
        frontier = src_nodes
    return blocks
