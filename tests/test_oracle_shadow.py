"""Pins for the oracle's ShaDow subgraph extraction (no GPU)."""
import numpy as np
import pytest

from oracle import model, sampling, shadow
from tests import helpers


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_shadow_components_brute_force(seed):
    rowptr, col = helpers.random_graph(64, 0.12, seed)
    A = helpers.dense_adjacency(rowptr, col)
    roots = np.random.Generator(np.random.PCG64(seed)).permutation(64)[:10]
    f, key = 3, 5 + seed
    blk, ptr = shadow.shadow_subgraphs(rowptr, col, roots, f, 2, key)
    B = len(roots)
    assert ptr[0] == B and ptr[-1] == blk.n_src == blk.n_dst
    assert np.array_equal(blk.src_nodes[:B], roots)
    for r, root in enumerate(roots):
        local = np.concatenate([[r], np.arange(ptr[r], ptr[r + 1])])
        nodes = blk.src_nodes[local]
        assert nodes[0] == root
        assert np.unique(nodes).shape[0] == nodes.shape[0]
        assert nodes.shape[0] <= 1 + f + f * f
        # brute force: hop 1 samples the root, hop 2 the nodes new at hop 1
        want = {int(root)}
        hop1 = [int(w) for w in sampling.sample_node(rowptr, col, int(root), f, key, 1)]
        new1 = [w for w in hop1 if w != root]
        want |= set(new1)
        for u in new1:
            want |= {int(w) for w in sampling.sample_node(rowptr, col, u, f, key, 2)}
        assert set(nodes.tolist()) == want
        # induced edges: exactly the adjacency restricted to the node set
        pos = {int(u): i for i, u in enumerate(local)}
        sub = np.zeros((nodes.shape[0], nodes.shape[0]))
        for i in local:
            row = blk.indices[blk.indptr[i]:blk.indptr[i + 1]]
            assert np.all(np.diff(blk.src_nodes[row]) > 0), "row not in ascending global order"
            for j in row:
                assert int(j) in pos, "edge leaves its component"
                sub[pos[int(i)], pos[int(j)]] += 1
        assert np.array_equal(sub, A[np.ix_(nodes, nodes)])
        assert np.array_equal(blk.src_nodes[blk.indices], blk.nbr)


def test_shadow_isolated_root_and_hub():
    rowptr, col = helpers.mixed_graph()
    blk, ptr = shadow.shadow_subgraphs(rowptr, col, np.array([51, 0]), 10, 2, 3)
    assert ptr.tolist()[:2] == [2, 2]           # isolated root: no other node, no edges
    assert blk.indptr[1] == 0
    assert blk.src_nodes[1] == 0 and ptr[2] - ptr[1] >= 10  # the hub and its sample


def test_shadow_train_step_readout_equals_root_rows():
    rowptr, col = helpers.random_graph(50, 0.15, 4)
    roots = np.array([4, 9, 31])
    X = np.random.Generator(np.random.PCG64(3)).normal(size=(50, 5))
    labels = np.random.Generator(np.random.PCG64(4)).integers(0, 3, 50)
    g = np.random.Generator(np.random.PCG64(5))
    ws = [g.normal(0, 0.5, s) for s in [(5, 4), (5, 4), (4, 3), (4, 3)]]
    res = shadow.shadow_train_step(rowptr, col, X, labels, roots, 3, 2, 7, model.SAGE_MEAN, ws, 0.0)
    assert np.array_equal(res["logits"], res["H"][-1][: len(roots)])
    # components are independent: one root alone gives the same logits row
    alone = shadow.shadow_train_step(rowptr, col, X, labels, roots[1:2], 3, 2, 7,
                                     model.SAGE_MEAN, ws, 0.0)
    assert np.allclose(alone["logits"][0], res["logits"][1], rtol=1e-13, atol=1e-13)


@pytest.mark.parametrize("kind,shapes", [
    (model.GCN, [(5, 4), (4, 3)]),
    (model.GIN, [(5, 4), (4, 4), (4, 3), (3, 3)]),      # W_a, W_b per layer
    (model.GAT, [(5, 4), (2, 4), (4, 3), (2, 3)]),      # W, a per layer
])
def test_shadow_train_step_layer_count_per_model(kind, shapes):
    # two layers whatever the number of matrices per layer: the logits have
    # the last layer's width, and one root alone gives its row of the batch
    rowptr, col = helpers.random_graph(50, 0.15, 4)
    roots = np.array([4, 9, 31])
    X = np.random.Generator(np.random.PCG64(3)).normal(size=(50, 5))
    labels = np.random.Generator(np.random.PCG64(4)).integers(0, 3, 50)
    g = np.random.Generator(np.random.PCG64(5))
    ws = [g.normal(0, 0.5, s) for s in shapes]
    res = shadow.shadow_train_step(rowptr, col, X, labels, roots, 3, 2, 7, kind, ws, 0.0)
    assert len(res["H"]) == 3 and res["logits"].shape == (3, 3)
    alone = shadow.shadow_train_step(rowptr, col, X, labels, roots[1:2], 3, 2, 7, kind, ws, 0.0)
    assert np.allclose(alone["logits"][0], res["logits"][1], rtol=1e-12, atol=1e-12)
