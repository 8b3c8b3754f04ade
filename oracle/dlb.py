"""Workload estimation and dynamic load balancing of mini-batches (CPU oracle).

Part of the CPU oracle (test infrastructure).

What the paper fixes (section 3, Dynamic Load Balancer): before training, the
sampling algorithm is run on every mini-batch and the number of aggregations
its computation graph needs is counted; that count is the batch's estimated
workload.  The batches are sorted by it, and each device receives batches
that add up to its share of the total workload (the workload ratio; a device
twice as fast gets twice the share).  After an epoch the measured execution
times are collected and, if the devices were imbalanced, the ratio is
recomputed from them.  Readings taken where the paper is silent:

* one aggregation is the addition of one feature element of one source row
  into one destination row: layer l runs on the block of hop L + 1 - l and
  costs (E + [GCN, GIN, GAT] n_dst) * width, E the block's sampled edges
  (GCN's normalised adjacency, GIN's sum and GAT's attention also take every
  destination row's own features, the self loop) and width the width of the
  rows it sums: dims[l - 1], or dims[l] for GAT (which sums transformed rows); ShaDow runs layers 1..L-1 on the union of the roots' subgraphs
  and layer L on the roots' rows only (its readout);
* assignment: batches in descending estimated workload (ties: lower batch
  index first), each to the worker whose assigned workload lies furthest
  below its target, ratio[j] / sum(ratio) * total (ties: lower worker
  index).  Every step gives the batch to a worker whose deficit is at least
  the mean remaining deficit, which is positive, so no worker ends more than
  one batch's workload above its target (and with two workers, none more
  than that below it);
* ratio update: a worker's speed is its assigned workload over its measured
  time, and the new ratio is proportional to speed.  Times within
  `tolerance` of each other (relative to the largest) count as balanced and
  keep the previous ratio.  A worker with no workload or no time keeps its
  previous share; the others divide the rest in proportion to speed.
"""
from __future__ import annotations

from typing import List, Sequence, Tuple

import numpy as np

from . import sampling, shadow


def layer_costs(kind: str, dims: Sequence[int], blocks_by_layer: List[Tuple[int, int]]) -> int:
    """sum over layers l of (E_l + [GCN, GIN, GAT] n_dst_l) * width_l (dims[l - 1],
    GAT dims[l]), given the (n_dst, E) of the block each layer runs on (layer
    order)."""
    assert kind in ("sage_mean", "gcn", "gin", "gat")
    total = 0
    for l, (n_dst, e) in enumerate(blocks_by_layer, start=1):
        terms = e + (n_dst if kind in ("gcn", "gin", "gat") else 0)
        total += int(terms) * int(dims[l] if kind == "gat" else dims[l - 1])
    return total


def estimate_work(rowptr, col, seeds_list, fanouts, keys, kind: str, dims: Sequence[int]):
    """Neighbour sampling: (work[n], edges[n, L]) for the batches seeds_list[i]
    sampled with keys[i] (the training step's blocks; edges[i, h] = E of hop
    h + 1)."""
    L = len(fanouts)
    assert len(dims) == L + 1
    n = len(seeds_list)
    work = np.zeros(n, dtype=np.int64)
    edges = np.zeros((n, L), dtype=np.int64)
    for i, (seeds, key) in enumerate(zip(seeds_list, keys)):
        blocks = sampling.sample_blocks(rowptr, col, seeds, fanouts, int(key))
        edges[i] = [b.n_edges for b in blocks]
        # layer l runs on hop L + 1 - l
        per_layer = [(blocks[L - l].n_dst, blocks[L - l].n_edges) for l in range(1, L + 1)]
        work[i] = layer_costs(kind, dims, per_layer)
    return work, edges


def shadow_estimate_work(rowptr, col, roots_list, fanout: int, hops: int, keys, kind: str,
                         dims: Sequence[int]):
    """ShaDow: (work[n], edges[n, 2]) with edges[i] = (edges of the union
    block, edges of the roots' rows)."""
    L = len(dims) - 1
    n = len(roots_list)
    work = np.zeros(n, dtype=np.int64)
    edges = np.zeros((n, 2), dtype=np.int64)
    for i, (roots, key) in enumerate(zip(roots_list, keys)):
        block, _ = shadow.shadow_subgraphs(rowptr, col, roots, fanout, hops, int(key))
        B = len(roots)
        e_root = int(block.indptr[B])
        edges[i] = (block.n_edges, e_root)
        per_layer = [(block.n_dst, block.n_edges)] * (L - 1) + [(B, e_root)]
        work[i] = layer_costs(kind, dims, per_layer)
    return work, edges


def assign(work, ratio) -> Tuple[np.ndarray, np.ndarray]:
    """(worker[n], load[k]): the greedy assignment of the module docstring."""
    work = [int(w) for w in work]
    ratio = [float(r) for r in ratio]
    k = len(ratio)
    assert k >= 1 and all(r >= 0 for r in ratio) and sum(ratio) > 0
    assert all(w >= 0 for w in work)
    total = sum(work)
    target = [r / sum(ratio) * total for r in ratio]
    load = [0] * k
    worker = [-1] * len(work)
    order = sorted(range(len(work)), key=lambda i: (-work[i], i))
    for i in order:
        best = 0
        for j in range(1, k):
            if target[j] - load[j] > target[best] - load[best]:
                best = j
        worker[i] = best
        load[best] += work[i]
    return np.array(worker, dtype=np.int64), np.array(load, dtype=np.int64)


def update_ratio(load, seconds, prev, tolerance: float) -> np.ndarray:
    """Next epoch's ratio (module docstring); the result sums to 1."""
    load = [float(x) for x in load]
    seconds = [float(x) for x in seconds]
    prev = [float(x) for x in prev]
    k = len(prev)
    assert len(load) == k and len(seconds) == k and sum(prev) > 0
    prev = [p / sum(prev) for p in prev]
    measured = [j for j in range(k) if load[j] > 0 and seconds[j] > 0]
    if not measured:
        return np.array(prev)
    times = [seconds[j] for j in measured]
    if max(times) - min(times) <= tolerance * max(times):
        return np.array(prev)
    speed = {j: load[j] / seconds[j] for j in measured}
    share = sum(prev[j] for j in measured)  # what the measured workers divide
    total_speed = sum(speed.values())
    out = list(prev)
    for j in measured:
        out[j] = share * speed[j] / total_speed
    return np.array(out)
