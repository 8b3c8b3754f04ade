"""Pins for the oracle's neighbour sampler and relabelling (no GPU)."""
import itertools
import math

import numpy as np
import pytest

from oracle import sampling
from tests import helpers


def _draw_for(t, m):
    """A 64-bit draw that the bounded map sends to exactly t in [0, m)."""
    return -(-(t << 64) // m)


@pytest.mark.parametrize("d,k", [(4, 2), (5, 3), (6, 3), (7, 4), (6, 5)])
def test_floyd_exhaustive_uniformity(d, k):
    # Every sequence (t_0..t_{k-1}) with t_s in [0, d-k+s] is equally likely;
    # Floyd's algorithm must map them onto each k-subset exactly k! times.
    ranges = [range(d - k + s + 1) for s in range(k)]
    counts = {}
    for ts in itertools.product(*ranges):
        draws = [_draw_for(t, d - k + s + 1) for s, t in enumerate(ts)]
        sub = tuple(sampling.floyd_positions(d, k, draws))
        assert len(set(sub)) == k and all(0 <= p < d for p in sub)
        assert list(sub) == sorted(sub)
        counts[sub] = counts.get(sub, 0) + 1
    assert len(counts) == math.comb(d, k)
    assert set(counts.values()) == {math.factorial(k)}


def test_floyd_chi_square_with_philox():
    # d = 6, k = 3 over many nodes: the 20 subsets must be equally frequent.
    rowptr, col = helpers.star_graph(6)  # node 0 has degree 6
    counts = {}
    n = 20000
    for key in range(n):
        sub = tuple(sampling.sample_node(rowptr, col, 0, 3, key + 1, 1))
        counts[sub] = counts.get(sub, 0) + 1
    assert len(counts) == 20
    exp = n / 20
    chi2 = sum((c - exp) ** 2 / exp for c in counts.values())
    assert chi2 < 50.0  # 19 dof; p ~ 1e-4


def _check_hop(rowptr, col, dst, f, indptr, nbr):
    for i, v in enumerate(dst):
        row = col[rowptr[v]:rowptr[v + 1]]
        got = nbr[indptr[i]:indptr[i + 1]]
        d = row.shape[0]
        assert got.shape[0] == min(f, d)
        assert np.unique(got).shape[0] == got.shape[0]
        assert np.all(np.isin(got, row))               # true neighbours
        assert np.all(np.diff(got) > 0)                 # ascending (= CSR order)
        if d <= f:
            assert np.array_equal(got, row)


@pytest.mark.parametrize("f", [1, 3, 5, 40, 64])
def test_sample_hop_invariants_and_scalar_reference(f):
    rowptr, col = helpers.mixed_graph()
    dst = np.arange(rowptr.shape[0] - 1)
    indptr, nbr = sampling.sample_hop(rowptr, col, dst, f, 7, 1)
    _check_hop(rowptr, col, dst, f, indptr, nbr)
    for i, v in enumerate(dst):
        ref = sampling.sample_node(rowptr, col, int(v), f, 7, 1)
        assert np.array_equal(nbr[indptr[i]:indptr[i + 1]], ref)


def test_sample_hop_random_graphs():
    for seed in range(5):
        rowptr, col = helpers.random_graph(60, 0.2, seed)
        g = np.random.Generator(np.random.PCG64(seed))
        dst = g.permutation(60)[:25]
        for f in (2, 5, 9):
            indptr, nbr = sampling.sample_hop(rowptr, col, dst, f, seed + 3, 2)
            _check_hop(rowptr, col, dst, f, indptr, nbr)
            for i, v in enumerate(dst):
                ref = sampling.sample_node(rowptr, col, int(v), f, seed + 3, 2)
                assert np.array_equal(nbr[indptr[i]:indptr[i + 1]], ref)


def test_inclusion_probability_hub():
    # Each of the 40 leaves of the hub is picked with probability k/d.
    rowptr, col = helpers.mixed_graph()
    hits = np.zeros(52)
    trials = 4000
    for key in range(trials):
        got = sampling.sample_node(rowptr, col, 0, 10, key, 1)
        hits[got] += 1
    p = hits[1:41] / trials
    assert np.all(np.abs(p - 0.25) < 0.035)


def test_keys_and_hops_change_the_sample():
    rowptr, col = helpers.mixed_graph()
    a = sampling.sample_node(rowptr, col, 0, 10, 1, 1)
    assert np.array_equal(a, sampling.sample_node(rowptr, col, 0, 10, 1, 1))
    assert not np.array_equal(a, sampling.sample_node(rowptr, col, 0, 10, 2, 1))
    assert not np.array_equal(a, sampling.sample_node(rowptr, col, 0, 10, 1, 2))


def test_relabel_matches_dictionary_scan():
    g = np.random.Generator(np.random.PCG64(9))
    for _ in range(50):
        nd = int(g.integers(0, 20))
        dst = g.permutation(100)[:nd]
        nbr = g.integers(0, 100, size=int(g.integers(0, 80)))
        s1, i1 = sampling.relabel(dst, nbr)
        s2, i2 = sampling.relabel_loop(dst, nbr)
        assert np.array_equal(s1, s2) and np.array_equal(i1, i2)
        assert np.array_equal(s1[:nd], dst)
        assert np.unique(s1).shape[0] == s1.shape[0]
        assert np.array_equal(s1[i1], nbr)


def test_relabel_worked_example():
    # dst (5, 2); edges 7, 2, 9, 7, 5, 3 -> src (5, 2, 7, 9, 3)
    s, i = sampling.relabel([5, 2], [7, 2, 9, 7, 5, 3])
    assert s.tolist() == [5, 2, 7, 9, 3]
    assert i.tolist() == [2, 1, 3, 2, 0, 4]


def test_sample_blocks_structure():
    rowptr, col = helpers.mixed_graph()
    seeds = np.array([0, 46, 51, 43])
    blocks = sampling.sample_blocks(rowptr, col, seeds, [5, 3, 2], 11)
    frontier = seeds
    for h, b in enumerate(blocks, start=1):
        assert b.hop == h
        assert np.array_equal(b.src_nodes[: b.n_dst], frontier)
        assert np.array_equal(b.src_nodes[b.indices], b.nbr)
        f = [5, 3, 2][h - 1]
        _check_hop(rowptr, col, frontier, f, b.indptr, b.nbr)
        assert b.n_src <= b.n_dst * (1 + f)
        frontier = b.src_nodes
    # node 51 is isolated: no edges
    assert blocks[0].indptr[3] == blocks[0].indptr[2]


def test_sub_batch_trees_are_identical():
    # Sampling is keyed by (key, hop, node): a seed's sampled neighbours are the
    # same whichever batch it is in.
    rowptr, col = helpers.random_graph(64, 0.15, 4)
    seeds = np.array([3, 17, 40, 22, 9, 58])
    full = sampling.sample_blocks(rowptr, col, seeds, [4, 3], 5)
    part = sampling.sample_blocks(rowptr, col, seeds[3:], [4, 3], 5)
    for i in range(3):
        a = full[0].nbr[full[0].indptr[3 + i]:full[0].indptr[4 + i]]
        b = part[0].nbr[part[0].indptr[i]:part[0].indptr[i + 1]]
        assert np.array_equal(a, b)
