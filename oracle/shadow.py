"""ShaDow k-hop localised subgraphs (CPU oracle).

Part of the CPU oracle (test infrastructure).

The paper (section 2.2, ShaDow K-Hop Sampling; section 5.2) runs an L-layer
GNN on a shallow subgraph localised around each root: the root's L'-hop
neighbourhood is neighbour-sampled, and all edges among the chosen node set
are kept (the subgraph is induced).  Readings taken:

* one subgraph per root; the batch is their disjoint union (a square block
  whose components do not touch), and the readout for a root is its own row;
* hops are taken breadth-first: hop h samples (with the same rule and Philox
  stream as neighbour sampling, counter word 2 = h) only the nodes first
  reached at hop h-1 (hop 1 samples the root);
* the node set of a root lists the root first, then the other nodes in order
  of first occurrence;
* local numbering of the union (a layout choice): the B roots take ids
  0..B-1 in batch order, then each component's other nodes follow, component
  after component, in their order of first occurrence; comp_ptr[r] is where
  component r's non-root nodes start and comp_ptr[B] the total;
* induced edges are listed per node in local-id order, and within a node in
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
    """Disjoint union of the roots' induced subgraphs, roots first.

    Returns (block, comp_ptr): block is square (n_dst == n_src == total nodes,
    src_nodes = global ids by local id, indices local); root r has local id r
    and component r's other nodes occupy [comp_ptr[r], comp_ptr[r+1])."""
    cache = {}
    B = len(roots)
    comps = [shadow_component(rowptr, col, int(r), fanout, hops, rng_key, cache) for r in roots]
    comp_ptr = [B]
    for nodes, _, _ in comps:
        comp_ptr.append(comp_ptr[-1] + nodes.shape[0] - 1)
    total = comp_ptr[-1]
    # local id of component-local index j of root r
    def to_local(r, j):
        return r if j == 0 else comp_ptr[r] + j - 1
    src_nodes = np.zeros(total, dtype=np.int64)
    row_edges = [None] * total
    for r, (nodes, counts, targets) in enumerate(comps):
        starts = np.concatenate([[0], np.cumsum(counts)])
        for j in range(nodes.shape[0]):
            u = to_local(r, j)
            src_nodes[u] = nodes[j]
            row_edges[u] = [to_local(r, int(t)) for t in targets[starts[j]:starts[j + 1]]]
    counts = np.array([len(e) for e in row_edges], dtype=np.int64)
    indptr = np.zeros(total + 1, dtype=np.int64)
    np.cumsum(counts, out=indptr[1:])
    indices = np.array([t for e in row_edges for t in e], dtype=np.int64)
    block = sampling.Block(0, indptr, indices, src_nodes, src_nodes[indices])
    return block, np.asarray(comp_ptr, dtype=np.int64)


def shadow_train_step(rowptr, col, X, labels, roots, fanout: int, hops: int, rng_key: int,
                      kind: str, weights, lr: float):
    """One ShaDow training step: every layer runs on the whole union subgraph and
    the loss reads out the root rows."""
    from . import model
    block, comp_ptr = shadow_subgraphs(rowptr, col, roots, fanout, hops, rng_key)
    L = len(weights) // (2 if kind in (model.SAGE_MEAN, model.GIN, model.GAT) else 1)
    xg = model.gather(X, block.src_nodes)
    y = np.asarray(labels)[np.asarray(roots, dtype=np.int64)]
    res = model.run_model(kind, weights, [block] * L, xg, y, lr, readout=np.arange(len(roots)),
                          bf16_layer1=model.is_bf16_features(X))
    res["block"] = block
    res["comp_ptr"] = comp_ptr
    res["xg"] = xg
    return res
