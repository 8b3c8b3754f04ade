"""Pins for the oracle's Philox4x64-10 stream and its bounded-integer map."""
import os

import numpy as np
import pytest

from oracle import philox, sampling

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "philox4x64_10_kat.txt")
M64 = (1 << 64) - 1


def _kat_rows():
    rows = []
    with open(GOLDEN) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            w = [int(x, 16) for x in line.split()]
            rows.append((tuple(w[0:4]), tuple(w[4:6]), tuple(w[6:10])))
    return rows


@pytest.mark.parametrize("ctr,key,expect", _kat_rows())
def test_philox_known_answers(ctr, key, expect):
    assert philox.philox4x64(ctr, key) == expect


@pytest.mark.parametrize("ctr,key,expect", _kat_rows())
def test_philox_vectorised_known_answers(ctr, key, expect):
    y = philox.philox4x64_vec(*[np.array([c], np.uint64) for c in ctr], key[0], key[1])
    assert tuple(int(v[0]) for v in y) == expect


@pytest.mark.parametrize("rng_key", [1, 2, 77, (1 << 63) + 5])
@pytest.mark.parametrize("hop", [1, 2, 3])
def test_stream_equals_numpy_philox(rng_key, hop):
    # numpy's Philox, started at counter (0, v, h, 0), is the library routine
    # the stream layout is defined against (it increments word 0 before a block).
    nodes = [0, 1, 5, 9999, 2_449_028, 110_999_999]
    got = philox.draws(rng_key, hop, np.array(nodes, np.uint64), 26)
    for i, v in enumerate(nodes):
        g = np.random.Philox(key=np.array([rng_key, 0], np.uint64),
                             counter=np.array([0, v, hop, 0], np.uint64))
        ref = g.random_raw(26)
        assert np.array_equal(got[i], ref)
        assert philox.draw_scalar(rng_key, hop, v, 13) == int(ref[13])


def test_bounded_closed_forms():
    assert sampling.bounded(0, 7) == 0
    assert sampling.bounded(M64, 7) == 6
    assert sampling.bounded(1 << 63, 10) == 5
    assert sampling.bounded(M64, 1) == 0
    # floor(r*m/2^64) for r = ceil(t*2^64/m) is exactly t
    for m in [1, 2, 3, 10, 1000, 123457, (1 << 31) - 1]:
        for t in {0, m // 2, m - 1}:
            r = -(-(t << 64) // m)
            assert sampling.bounded(r, m) == t


def test_bounded_vectorised_matches_python_ints():
    g = np.random.Generator(np.random.PCG64(5))
    r = g.integers(0, 1 << 64, size=5000, dtype=np.uint64)
    m = g.integers(1, 1 << 32, size=5000, dtype=np.uint64)
    got = sampling.bounded_vec(r, m)
    ref = np.array([(int(a) * int(b)) >> 64 for a, b in zip(r, m)], np.int64)
    assert np.array_equal(got, ref)
    assert np.all(got < m.astype(np.int64))


def test_bounded_is_nearly_uniform():
    g = np.random.Generator(np.random.PCG64(6))
    r = g.integers(0, 1 << 64, size=200_000, dtype=np.uint64)
    t = sampling.bounded_vec(r, np.full(r.shape, 7, np.uint64))
    counts = np.bincount(t, minlength=7)
    expected = r.shape[0] / 7
    chi2 = ((counts - expected) ** 2 / expected).sum()
    assert chi2 < 30.0  # 6 dof; p ~ 4e-5
