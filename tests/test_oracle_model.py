"""Pins for the oracle's aggregation, forward, loss, backward and SGD (no GPU)."""
import math

import numpy as np
import pytest

from oracle import model, sampling
from tests import helpers


def _full_blocks(rowptr, col, order, L):
    """Every node a seed and budgets >= max degree: all L blocks are the whole graph."""
    blocks = sampling.sample_blocks(rowptr, col, order, [64] * L, 3)
    for b in blocks:
        assert b.n_src == b.n_dst == order.shape[0]
    return blocks


def _weights(kind, dims, seed):
    g = np.random.Generator(np.random.PCG64(seed))
    ws = []
    for l in range(1, len(dims)):
        if kind == model.GAT:   # W [F_{l-1} x F_l], attention vectors a [2 x F_l]
            ws.append(g.normal(0, 1.0 / math.sqrt(dims[l - 1]), (dims[l - 1], dims[l])))
            ws.append(g.normal(0, 1.0, (2, dims[l])))
            continue
        if kind == model.GIN:   # the MLP: W_a [F_{l-1} x F_l], W_b [F_l x F_l]
            ws.append(g.normal(0, 1.0 / math.sqrt(dims[l - 1]), (dims[l - 1], dims[l])))
            ws.append(g.normal(0, 1.0 / math.sqrt(dims[l]), (dims[l], dims[l])))
            continue
        for _ in range(2 if kind == model.SAGE_MEAN else 1):
            ws.append(g.normal(0, 1.0 / math.sqrt(dims[l - 1]), (dims[l - 1], dims[l])))
    return ws


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_sage_mean_equals_dense_row_normalised_adjacency(seed):
    rowptr, col = helpers.random_graph(40, 0.12, seed)
    A = helpers.dense_adjacency(rowptr, col)
    order = np.random.Generator(np.random.PCG64(seed)).permutation(40)
    blk = _full_blocks(rowptr, col, order, 1)[0]
    deg = A.sum(1)
    Dinv = np.where(deg > 0, 1.0 / np.maximum(deg, 1), 0.0)
    ref = (Dinv[:, None] * A)[np.ix_(order, order)]
    got = model.agg_matrix(blk, model.SAGE_MEAN).toarray()
    assert np.allclose(got, ref, rtol=0, atol=1e-15)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_gcn_equals_kipf_normalisation(seed):
    rowptr, col = helpers.random_graph(40, 0.12, seed)
    A = helpers.dense_adjacency(rowptr, col)
    order = np.random.Generator(np.random.PCG64(seed + 10)).permutation(40)
    blk = _full_blocks(rowptr, col, order, 1)[0]
    At = A + np.eye(40)
    dt = At.sum(1)
    ref = (At / np.sqrt(np.outer(dt, dt)))[np.ix_(order, order)]
    got = model.agg_matrix(blk, model.GCN).toarray()
    assert np.allclose(got, ref, rtol=0, atol=1e-15)


def test_mean_of_constant_and_regular_gcn_row_sums():
    rowptr, col = helpers.mixed_graph()
    blocks = sampling.sample_blocks(rowptr, col, np.array([0, 41, 51, 46]), [7, 3], 2)
    for b in blocks:
        H = np.full((b.n_src, 3), 2.5)
        agg = model.agg_matrix(b, model.SAGE_MEAN) @ H
        c = np.diff(b.indptr)
        assert np.allclose(agg[c > 0], 2.5) and np.all(agg[c == 0] == 0)
    # GCN on a d-regular graph, full case: Ahat 1 = 1
    for rp, cl, n in [(*helpers.complete_graph(5), 5), (*helpers.cycle_graph(9), 9)]:
        blk = _full_blocks(rp, cl, np.arange(n)[::-1].copy(), 1)[0]
        assert np.allclose(model.agg_matrix(blk, model.GCN) @ np.ones(n), 1.0)


def test_gcn_out_degree_counts_self_edge():
    s, idx = sampling.relabel([4, 6], [6, 9, 9, 4, 1])
    b = sampling.Block(1, np.array([0, 3, 5]), idx, s, s[idx])
    # src = (4, 6, 9, 1); edges into 6 once, 9 twice, 4 once, 1 once; +1 for dst 4 and 6
    assert model.out_degree(b).tolist() == [2, 2, 2, 1]


def _dense_gat(A, H, W, a):
    # every node attends over its closed neighbourhood: a masked dense softmax
    T = H @ W
    E = (T @ a[0])[:, None] + (T @ a[1])[None, :]
    E = np.where(E > 0, E, 0.2 * E)
    E = np.where(A + np.eye(len(A)) > 0, E, -np.inf)
    P = np.exp(E - E.max(1, keepdims=True))
    return (P / P.sum(1, keepdims=True)) @ T


@pytest.mark.parametrize("kind", [model.SAGE_MEAN, model.GCN, model.GIN, model.GAT])
def test_forward_equals_full_graph_dense_gnn(kind):
    rowptr, col = helpers.random_graph(30, 0.15, 7)
    A = helpers.dense_adjacency(rowptr, col)
    order = np.random.Generator(np.random.PCG64(1)).permutation(30)
    dims = (6, 5, 4, 3)
    blocks = _full_blocks(rowptr, col, order, 3)
    g = np.random.Generator(np.random.PCG64(2))
    X = g.normal(size=(30, 6))
    ws = _weights(kind, dims, 3)
    y = g.integers(0, 3, 30)
    res = model.run_model(kind, ws, blocks[::-1], X[order], y[order], 0.0)
    # dense full-batch model on the original node order
    deg = A.sum(1)
    if kind == model.SAGE_MEAN:
        Ahat = np.where(deg[:, None] > 0, A / np.maximum(deg, 1)[:, None], 0.0)
    elif kind == model.GIN:
        Ahat = A + np.eye(30)   # GIN-0: (1 + 0) h_v + sum of the neighbours
    else:
        At = A + np.eye(30)
        Ahat = At / np.sqrt(np.outer(At.sum(1), At.sum(1)))
    H = X
    for l in range(1, 4):
        if kind == model.SAGE_MEAN:
            Z = H @ ws[2 * l - 2] + Ahat @ H @ ws[2 * l - 1]
        elif kind == model.GIN:
            Z = np.maximum(Ahat @ H @ ws[2 * l - 2], 0) @ ws[2 * l - 1]
        elif kind == model.GAT:
            Z = _dense_gat(A, H, ws[2 * l - 2], ws[2 * l - 1])
        else:
            Z = Ahat @ H @ ws[l - 1]
        H = np.maximum(Z, 0) if l < 3 else Z
    assert np.allclose(res["logits"], H[order], rtol=1e-12, atol=1e-12)


def test_loss_closed_form_zero_last_layer():
    rowptr, col = helpers.random_graph(50, 0.1, 3)
    seeds = np.arange(0, 50, 3)
    blocks = sampling.sample_blocks(rowptr, col, seeds, [4, 3], 9)
    dims = (5, 7, 16)
    ws = _weights(model.SAGE_MEAN, dims, 1)
    ws[2][:] = 0
    ws[3][:] = 0
    X = np.random.Generator(np.random.PCG64(0)).normal(size=(blocks[-1].n_src, 5))
    res = model.run_model(model.SAGE_MEAN, ws, blocks[::-1], X, np.zeros(len(seeds), int), 0.1)
    assert abs(res["loss"] - math.log(16)) < 1e-14
    # gradient of the loss w.r.t. logits of a uniform prediction: (1/C - onehot)/B
    d = res["dlogits"]
    assert np.allclose(d[:, 0], (1 / 16 - 1) / len(seeds)) and np.allclose(d[:, 1:], 1 / 16 / len(seeds))


def _problem(kind, seed):
    rowptr, col = helpers.random_graph(60, 0.1, seed)
    seeds = np.random.Generator(np.random.PCG64(seed)).permutation(60)[:12]
    blocks = sampling.sample_blocks(rowptr, col, seeds, [5, 4, 3], seed + 1)
    dims = (4, 6, 5, 3)
    g = np.random.Generator(np.random.PCG64(seed + 2))
    X = g.normal(size=(blocks[-1].n_src, 4))
    y = g.integers(0, 3, len(seeds))
    return blocks, X, y, _weights(kind, dims, seed + 3)


@pytest.mark.parametrize("kind", [model.SAGE_MEAN, model.GCN, model.GIN, model.GAT])
def test_gradients_central_finite_differences(kind):
    # an instance whose hidden pre-activations all sit clear of the ReLU kinks
    # (checked below; for GIN seed 5 has one within 3e-5 of 0, for GAT an
    # all-zero hidden row whose self-edge score is exactly 0)
    blocks, X, y, ws = _problem(kind, 9 if kind in (model.GIN, model.GAT) else 5)
    res = model.run_model(kind, ws, blocks[::-1], X, y, 0.0)
    if kind == model.GAT:
        # and every attention score clear of LeakyReLU's kink
        for l, blk in enumerate(blocks[::-1], start=1):
            _, c = model.gat_forward(blk, res["H"][l - 1], ws[2 * l - 2], ws[2 * l - 1])
            assert np.abs(c["pre"]).min() > 1e-4
    # (a GIN row whose MLP hidden row is all zero has Z exactly 0 there, and
    # stays 0 under the perturbations below)
    for P in res["P"]:
        assert np.abs(P).min() > 1e-4
    for Z in res["Z"][:-1]:
        assert np.abs(Z[Z != 0]).min() > 1e-4
    h = 1e-6
    g = np.random.Generator(np.random.PCG64(0))
    for wi, W in enumerate(ws):
        for _ in range(6):
            i, j = g.integers(0, W.shape[0]), g.integers(0, W.shape[1])
            wp = [w.copy() for w in ws]
            wm = [w.copy() for w in ws]
            wp[wi][i, j] += h
            wm[wi][i, j] -= h
            lp = model.run_model(kind, wp, blocks[::-1], X, y, 0.0)["loss"]
            lm = model.run_model(kind, wm, blocks[::-1], X, y, 0.0)["loss"]
            fd = (lp - lm) / (2 * h)
            an = res["dW"][wi][i, j]
            assert abs(fd - an) <= 1e-6 * max(1.0, abs(an)), (wi, i, j, fd, an)


@pytest.mark.parametrize("kind", [model.SAGE_MEAN])
def test_sync_sgd_equivalence_of_sub_batches(kind):
    # Gradients of the full batch equal the size-weighted mean of the sub-batch
    # gradients (sampling is keyed per node, so every seed's tree is unchanged).
    # Only GraphSAGE-mean has per-seed independent gradients: the GCN weights use
    # block-level out-degrees, which depend on the other seeds of the batch
    # (see test_gcn_block_normalisation_couples_seeds).
    rowptr, col = helpers.random_graph(64, 0.1, 8)
    seeds = np.random.Generator(np.random.PCG64(8)).permutation(64)[:16]
    dims = (4, 6, 3)
    ws = _weights(kind, dims, 9)
    X = np.random.Generator(np.random.PCG64(1)).normal(size=(64, 4))
    labels = np.random.Generator(np.random.PCG64(2)).integers(0, 3, 64)
    full = model.train_step(rowptr, col, X, labels, seeds, [5, 3], 4, kind, ws, 0.0)
    acc = [np.zeros_like(w) for w in ws]
    loss = 0.0
    for part in (seeds[:5], seeds[5:11], seeds[11:]):
        r = model.train_step(rowptr, col, X, labels, part, [5, 3], 4, kind, ws, 0.0)
        for a, g in zip(acc, r["dW"]):
            a += g * len(part) / len(seeds)
        loss += r["loss"] * len(part) / len(seeds)
    assert abs(loss - full["loss"]) < 1e-12
    for a, g in zip(acc, full["dW"]):
        assert np.allclose(a, g, rtol=1e-10, atol=1e-13)


def test_sgd_step_decreases_loss():
    blocks, X, y, ws = _problem(model.SAGE_MEAN, 2)
    r0 = model.run_model(model.SAGE_MEAN, ws, blocks[::-1], X, y, 1e-3)
    for w, w1, g in zip(ws, r0["W_new"], r0["dW"]):
        assert np.array_equal(w1, w - 1e-3 * g)
    r1 = model.run_model(model.SAGE_MEAN, r0["W_new"], blocks[::-1], X, y, 0.0)
    gn = sum(float((g * g).sum()) for g in r0["dW"])
    assert r1["loss"] < r0["loss"] - 0.5e-3 * gn


def test_bf16_widening_is_exact():
    bits = np.array([[0x3F80, 0xC000, 0x3FC0, 0x0000, 0x8000, 0x4049]], np.uint16)
    got = model.widen(bits)
    assert got[0, :5].tolist() == [1.0, -2.0, 1.5, 0.0, -0.0]
    assert got[0, 5] == 3.140625


def test_gcn_block_normalisation_couples_seeds():
    # The condition of the sync-SGD equivalence (independent per-seed gradients)
    # does not hold for block-normalised GCN: adding seeds changes d_out.
    s, idx = sampling.relabel([1], [5, 6])
    one = sampling.Block(1, np.array([0, 2]), idx, s, s[idx])
    s2, idx2 = sampling.relabel([1, 2], [5, 6, 5])
    two = sampling.Block(1, np.array([0, 2, 3]), idx2, s2, s2[idx2])
    a1 = model.agg_matrix(one, model.GCN).toarray()[0]
    a2 = model.agg_matrix(two, model.GCN).toarray()[0]
    assert a1[1] != a2[2]  # weight of edge (1 -> 5) changes with the batch


def test_gat_without_attention_is_the_closed_neighbourhood_mean():
    # a = 0: every edge scores 0, so v averages T over N(v) + {v}
    rowptr, col = helpers.random_graph(40, 0.1, 4)
    seeds = np.arange(0, 40, 2)
    blk = sampling.sample_blocks(rowptr, col, seeds, [3], 5)[0]
    g = np.random.Generator(np.random.PCG64(4))
    H = g.normal(size=(blk.n_src, 5))
    W = g.normal(size=(5, 3))
    out, c = model.gat_forward(blk, H, W, np.zeros((2, 3)))
    T = H @ W
    for v in range(blk.n_dst):
        nb = list(blk.indices[blk.indptr[v]: blk.indptr[v + 1]]) + [v]
        assert np.allclose(out[v], T[nb].mean(0), rtol=1e-13, atol=1e-13)
    # the attention weights of each row sum to 1
    assert np.allclose(np.bincount(c["rows"], weights=c["alpha"]), 1.0)


def test_gat_isolated_node_keeps_its_own_row():
    # a dst node with no sampled edge attends to itself only: out_v = T_v
    rowptr = np.array([0, 0, 1, 2], dtype=np.int64)   # node 0 isolated, 1 - 2
    col = np.array([2, 1], dtype=np.int32)
    blk = sampling.sample_blocks(rowptr, col, np.array([0, 1]), [4], 1)[0]
    assert blk.indptr.tolist() == [0, 0, 1]
    g = np.random.Generator(np.random.PCG64(1))
    H = g.normal(size=(blk.n_src, 4))
    W = g.normal(size=(4, 2))
    a = g.normal(size=(2, 2))
    out, _ = model.gat_forward(blk, H, W, a)
    assert np.allclose(out[0], (H @ W)[0], rtol=1e-14, atol=1e-14)
    # node 1 mixes itself and node 2 with the logistic weight of the score gap
    T = H @ W
    e = [a[0] @ T[1] + a[1] @ T[u] for u in (1, 2)]
    e = [x if x > 0 else 0.2 * x for x in e]
    w2 = 1.0 / (1.0 + math.exp(e[0] - e[1]))
    assert np.allclose(out[1], (1 - w2) * T[1] + w2 * T[2], rtol=1e-12, atol=1e-12)


def test_gin_sums_neighbours_and_self():
    # constant features: a dst row's aggregation is (sampled edges + 1) times the constant
    rowptr, col = helpers.mixed_graph()
    seeds = np.array([0, 46, 51, 43])
    blk = sampling.sample_blocks(rowptr, col, seeds, [5], 2)[0]
    A = model.agg_matrix(blk, model.GIN)
    agg = A @ np.full((blk.n_src, 3), 2.0)
    np.testing.assert_array_equal(agg[:, 0], 2.0 * (np.diff(blk.indptr) + 1))
