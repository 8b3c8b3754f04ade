"""Pins for the oracle's workload estimate and dynamic load balancer (no GPU).

Expected values below are worked out by hand from the definitions (section 3,
Dynamic Load Balancer, with the readings stated in oracle/dlb.py); none comes
from the oracle itself."""
import itertools

import numpy as np
import pytest

from oracle import dlb
from tests import helpers


def _ball(rowptr, col, seeds, radius):
    """Nodes within `radius` hops of the seeds (brute force over the CSR)."""
    ball = set(int(s) for s in seeds)
    for _ in range(radius):
        ball |= {int(w) for v in ball for w in col[rowptr[v]:rowptr[v + 1]]}
    return ball


def test_work_of_a_path_by_hand():
    # path 0-1-2-3, seed 0, budgets above every degree (whole neighbourhoods):
    # hop 1: dst {0}, E = deg 0 = 1; hop 2: dst {0, 1}, E = 1 + 2 = 3.
    # dims (4, 3, 2): layer 1 runs on hop 2, layer 2 on hop 1.
    #   SAGE-mean: 3 * 4 + 1 * 3 = 15
    #   GCN and GIN (self loops): (3 + 2) * 4 + (1 + 1) * 3 = 26
    rowptr, col = helpers.path_graph(4)
    #   GAT sums transformed rows (width dims[l]): (3 + 2) * 3 + (1 + 1) * 2 = 19
    for kind, want in (("sage_mean", 15), ("gcn", 26), ("gin", 26), ("gat", 19)):
        work, edges = dlb.estimate_work(rowptr, col, [np.array([0])], [5, 5], [7], kind, (4, 3, 2))
        assert work.tolist() == [want], kind
        assert edges.tolist() == [[1, 3]]


def test_shadow_work_of_a_path_by_hand():
    # path 0-1-2-3, root 0, fanout 5, 2 hops: node set {0, 1, 2}; induced
    # edges 0-1, 1-0, 1-2, 2-1 (E = 4), the root's row holds 1 of them.
    # dims (4, 3, 2): layer 1 on the union, layer 2 on the root row.
    #   SAGE-mean: 4 * 4 + 1 * 3 = 19;  GCN, GIN: (4 + 3) * 4 + (1 + 1) * 3 = 34
    rowptr, col = helpers.path_graph(4)
    #   GAT (widths dims[l]): (4 + 3) * 3 + (1 + 1) * 2 = 25
    for kind, want in (("sage_mean", 19), ("gcn", 34), ("gin", 34), ("gat", 25)):
        work, edges = dlb.shadow_estimate_work(rowptr, col, [np.array([0])], 5, 2, [3], kind,
                                               (4, 3, 2))
        assert work.tolist() == [want], kind
        assert edges.tolist() == [[4, 1]]


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_whole_neighbourhoods_count_the_bfs_balls(seed):
    # with budgets above every degree each hop keeps every edge of its
    # frontier: hop h has the ball of radius h - 1 as dst nodes and the sum of
    # their degrees as edges
    rowptr, col = helpers.random_graph(60, 0.08, seed)
    deg = np.diff(rowptr)
    seeds = np.random.Generator(np.random.PCG64(seed)).permutation(60)[:5]
    fan = [64, 64, 64]
    dims = (6, 5, 4, 3)
    work, edges = dlb.estimate_work(rowptr, col, [seeds], fan, [seed + 1], "gcn", dims)
    want_e, want_n = [], []
    for h in range(1, 4):
        ball = _ball(rowptr, col, seeds, h - 1)
        want_n.append(len(ball))
        want_e.append(int(sum(deg[v] for v in ball)))
    assert edges[0].tolist() == want_e
    want_work = sum((want_e[3 - l] + want_n[3 - l]) * dims[l - 1] for l in range(1, 4))
    assert int(work[0]) == want_work


def test_budgets_bound_the_edges():
    rowptr, col = helpers.mixed_graph()
    deg = np.diff(rowptr)
    batches = [np.array([0, 46, 51]), np.array([41, 3])]
    work, edges = dlb.estimate_work(rowptr, col, batches, [4, 2], [11, 12], "sage_mean", (8, 8, 4))
    # hop 1: min(budget, degree) per seed
    for i, seeds in enumerate(batches):
        assert edges[i, 0] == sum(min(4, int(deg[s])) for s in seeds)
    assert work.tolist() == [int(edges[i, 1]) * 8 + int(edges[i, 0]) * 8 for i in range(2)]


def test_assign_by_hand():
    # targets 15 / 15; descending: 10 -> w0 (tie), 9 -> w1, 8 -> w1 (deficits
    # 5 < 6), then each 1 -> w0 (5 > -2): loads 13 / 17
    worker, load = dlb.assign([10, 9, 8, 1, 1, 1], [1, 1])
    assert worker.tolist() == [0, 1, 1, 0, 0, 0]
    assert load.tolist() == [13, 17]
    # a third of equal batches: 9 batches of 1 with ratio 1 : 2 -> 3 and 6
    worker, load = dlb.assign([1] * 9, [1, 2])
    assert load.tolist() == [3, 6]
    assert worker.tolist() == [1, 1, 1, 0, 1, 0, 1, 0, 1]


def test_assign_ties_and_zero_ratio():
    # equal work: batch order decides; a worker with ratio 0 gets nothing
    worker, load = dlb.assign([5, 5, 5, 5], [0, 1, 1])
    assert worker.tolist() == [1, 2, 1, 2]
    assert load.tolist() == [0, 10, 10]
    worker, load = dlb.assign([], [1, 1])
    assert worker.tolist() == [] and load.tolist() == [0, 0]


@pytest.mark.parametrize("seed", range(6))
def test_assign_bounds(seed):
    g = np.random.Generator(np.random.PCG64(seed))
    n, k = int(g.integers(1, 40)), int(g.integers(1, 5))
    work = g.integers(0, 1000, n) if seed % 2 else (g.pareto(1.5, n) * 100).astype(np.int64)
    ratio = g.random(k) + 0.05
    worker, load = dlb.assign(work, ratio)
    assert sorted(set(worker.tolist())) <= list(range(k))
    for j in range(k):
        assert load[j] == int(work[worker == j].sum())
    total, wmax = int(work.sum()), int(work.max())
    target = ratio / ratio.sum() * total
    assert np.all(load - target <= wmax + 1e-9)          # never a batch above target
    if k == 2:
        assert np.all(np.abs(load - target) <= wmax + 1e-9)


def test_assign_two_workers_matches_exhaustive_search_on_small_sets():
    # greedy is a heuristic; on these sets it reaches the best split
    for work in ([10, 9, 8, 1, 1, 1], [7, 5, 4, 3, 1], [6, 6, 4, 4, 2, 2]):
        _, load = dlb.assign(work, [1, 1])
        best = min(abs(sum(c) - (sum(work) - sum(c)))
                   for r in range(len(work) + 1) for c in itertools.combinations(work, r))
        assert abs(int(load[0]) - int(load[1])) == best


def test_update_ratio_closed_forms():
    # speeds 100 / 150 -> 2 : 3
    np.testing.assert_allclose(dlb.update_ratio([100, 300], [1.0, 2.0], [0.5, 0.5], 0.05),
                               [0.4, 0.6])
    # equal times are balanced whatever the loads: the ratio stays
    np.testing.assert_allclose(dlb.update_ratio([100, 300], [1.0, 1.0], [0.5, 0.5], 0.0),
                               [0.5, 0.5])
    # equal times within the tolerance keep the previous ratio
    np.testing.assert_allclose(dlb.update_ratio([100, 300], [1.0, 1.02], [0.4, 0.6], 0.05),
                               [0.4, 0.6])
    # an idle worker keeps its share, the others divide the rest by speed
    np.testing.assert_allclose(dlb.update_ratio([0, 100, 200], [0, 1.0, 4.0], [0.5, 0.25, 0.25],
                                                0.0), [0.5, 0.5 * 2 / 3, 0.5 / 3])
    # a balanced outcome is a fixed point: workload proportional to speed
    r = dlb.update_ratio([200, 600], [2.0, 3.0], [0.5, 0.5], 0.0)
    np.testing.assert_allclose(r, [100 / 300, 200 / 300])
    np.testing.assert_allclose(dlb.update_ratio([200 * r[0], 200 * r[1]], [1.0, 1.0], r, 0.0), r)
