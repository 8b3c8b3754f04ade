"""ShaDow k-hop localised subgraphs (CPU oracle).

Part of the CPU oracle (test infrastructure).

The paper (section 2.2, ShaDow K-Hop Sampling; section 5.2) runs an L-layer
GNN on a shallow subgraph localised around each root: the root's L'-hop
neighbourhood is neighbour-sampled, and all edges among the chosen node set
are kept (the subgraph is induced).  Readings taken:

* one subgraph per root; the batch is their disjoint union (a block-diagonal
  square block), and the readout for a root is its own row;
* hops are taken breadth-first: hop h samples (with the same rule and Philox
  stream as neighbour sampling, counter word 2 = h) only the nodes first
  reached at hop h-1 (hop 1 samples the root);
* the node set of a root lists the root first, then the other nodes in order
  of first occurrence;
* induced edges are listed per node in local order, and within a node in
  ascending global neighbour id (CSR order).
"""
from __future__ import annotations

import numpy as np

from . import sampling


def shadow_component(rowptr, col, root: int, fanout: int, hops: int, rng_key: int, cache=None):
    """Node list (global ids, first-occurrence order) and induced edges of one root."""
    cache = {} if cache is None else cache
    nodes = [int(root)]
    local = {int(root): 0}
    frontier = [int(root)]
    for h in range(1, hops + 1):
        reached = []
        for u in frontier:
            key = (u, h)
            if key not in cache:
                cache[key] = sampling.sample_node(rowptr, col, u, fanout, rng_key, h)
            for w in cache[key]:
                w = int(w)
                if w not in local:
                    local[w] = len(nodes)
                    nodes.append(w)
                    reached.append(w)
        frontier = reached
    node_arr = np.asarray(nodes, dtype=np.int64)
    counts, targets = [], []
    for u in nodes:
        row = np.asarray(col[int(rowptr[u]):int(rowptr[u + 1])], dtype=np.int64)
        keep = row[np.isin(row, node_arr)]
        counts.append(keep.shape[0])
        targets.extend(local[int(w)] for w in keep)
    return node_arr, np.asarray(counts, np.int64), np.asarray(targets, np.int64)


def shadow_subgraphs(rowptr, col, roots, fanout: int, hops: int, rng_key: int):
    """Block-diagonal union of the roots' induced subgraphs.

    Returns (block, comp_ptr): block is square (n_dst == n_src == total nodes,
    src_nodes = concatenated node lists, indices local to the union), and the
    nodes of root r occupy [comp_ptr[r], comp_ptr[r+1]) with the root first."""
    cache = {}
    comp_ptr = [0]
    all_nodes, all_counts, all_idx = [], [], []
    for r in roots:
        nodes, counts, targets = shadow_component(rowptr, col, int(r), fanout, hops, rng_key, cache)
        off = comp_ptr[-1]
        all_nodes.append(nodes)
        all_counts.append(counts)
        all_idx.append(targets + off)
        comp_ptr.append(off + nodes.shape[0])
    nodes = np.concatenate(all_nodes) if all_nodes else np.zeros(0, np.int64)
    counts = np.concatenate(all_counts) if all_counts else np.zeros(0, np.int64)
    indices = np.concatenate(all_idx) if all_idx else np.zeros(0, np.int64)
    indptr = np.zeros(nodes.shape[0] + 1, dtype=np.int64)
    np.cumsum(counts, out=indptr[1:])
    block = sampling.Block(0, indptr, indices, nodes, nodes[indices])
    return block, np.asarray(comp_ptr, dtype=np.int64)


def shadow_train_step(rowptr, col, X, labels, roots, fanout: int, hops: int, rng_key: int,
                      kind: str, weights, lr: float):
    """One ShaDow training step: every layer runs on the whole union subgraph and
    the loss reads out the root rows."""
    from . import model
    block, comp_ptr = shadow_subgraphs(rowptr, col, roots, fanout, hops, rng_key)
    L = len(weights) // (2 if kind == model.SAGE_MEAN else 1)
    xg = model.gather(X, block.src_nodes)
    y = np.asarray(labels)[np.asarray(roots, dtype=np.int64)]
    res = model.run_model(kind, weights, [block] * L, xg, y, lr, readout=comp_ptr[:-1])
    res["block"] = block
    res["comp_ptr"] = comp_ptr
    res["xg"] = xg
    return res
