"""Pins for the oracle's GPU feature cache (no GPU).  Expected values are
worked out by hand or come from a textbook LRU; none comes from the oracle."""
from collections import OrderedDict

import numpy as np
import pytest

from oracle import feature_cache as fc


def test_fmix32_known_answers():
    # MurmurHash3_x86_32 of an empty key is fmix32(seed); published test
    # vectors: seed 0 -> 0, seed 1 -> 0x514E28B7, seed 0xFFFFFFFF -> 0x81F16F39
    assert fc.fmix32(0) == 0
    assert fc.fmix32(1) == 0x514E28B7
    assert fc.fmix32(0xFFFFFFFF) == 0x81F16F39


def test_fmix32_is_a_bijection_on_a_sample():
    vals = [fc.fmix32(v) for v in range(0, 1 << 20, 3)]
    assert len(set(vals)) == len(vals)
    assert all(0 <= h <= 0xFFFFFFFF for h in vals[:1000])


def _table(n, F=3):
    return np.arange(n * F, dtype=np.float32).reshape(n, F)


def test_lru_by_hand():
    # one set, two ways; one node per call
    X = _table(20)
    c = fc.FeatureCache(1, 2, 3)
    hits = [c.fetch(X, [v])[1] for v in (5, 6, 5, 7, 6)]
    # 5 miss (in), 6 miss (in), 5 hit, 7 miss evicts 6 (stamp 2 < 3), 6 miss evicts 5
    assert hits == [0, 0, 1, 0, 0]
    assert set(c.contents()) == {7, 6}


def test_overflowing_set_keeps_request_order():
    X = _table(20)
    c = fc.FeatureCache(1, 2, 3)
    out, h, m = c.fetch(X, [10, 11, 12])
    assert (h, m) == (0, 3)
    np.testing.assert_array_equal(out, X[[10, 11, 12]])
    assert set(c.contents()) == {10, 11}          # the first two misses, in request order
    out, h, m = c.fetch(X, [12, 11])
    assert (h, m) == (1, 1)
    # 11 was read by this call; 10 (stamp 1) is the only replaceable entry
    assert c.contents() == {12: (0, 0, 2), 11: (0, 1, 2)}


def test_entries_read_in_a_call_are_not_replaced_by_it():
    X = _table(40)
    c = fc.FeatureCache(1, 3, 3)
    c.fetch(X, [1, 2, 3])
    _, h, m = c.fetch(X, [1, 2, 3, 4, 5])
    assert (h, m) == (3, 2)
    assert set(c.contents()) == {1, 2, 3}         # no entry older than this call


@pytest.mark.parametrize("ways", [1, 2, 4, 8])
def test_single_node_calls_equal_a_textbook_lru(ways):
    # with one set and one node per call, recency in calls is plain LRU
    g = np.random.Generator(np.random.PCG64(ways))
    X = _table(30)
    c = fc.FeatureCache(1, ways, 3)
    lru = OrderedDict()
    for v in g.integers(0, 30, 400):
        v = int(v)
        _, h, _ = c.fetch(X, [v])
        want = v in lru
        assert h == int(want)
        if want:
            lru.move_to_end(v)
        else:
            lru[v] = True
            if len(lru) > ways:
                lru.popitem(last=False)
        assert set(c.contents()) == set(lru)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_rows_and_invariants(seed):
    g = np.random.Generator(np.random.PCG64(seed))
    X = g.normal(size=(500, 4)).astype(np.float32)
    c = fc.FeatureCache(7, 4, 4)
    total_hits = 0
    for call in range(30):
        ids = g.choice(500, size=int(g.integers(1, 80)), replace=False) if call % 3 else \
            g.choice(60, size=20, replace=False)   # a hot subset recurs
        out, h, m = c.fetch(X, ids)
        np.testing.assert_array_equal(out, X[ids])
        assert h + m == len(ids)
        total_hits += h
        cont = c.contents()
        assert len(cont) == len({k for k in cont})   # no node cached twice
        for v, (s, w, st) in cont.items():
            assert fc.set_of(v, 7) == s and 1 <= st <= call + 1
            np.testing.assert_array_equal(c.rows[s, w], X[v])
        for v in ids:
            if int(v) in cont:
                assert cont[int(v)][2] == call + 1       # read or inserted by this call
    assert total_hits > 0
