"""The load balancer's host entry points (gnn_dlb_assign, gnn_dlb_ratio)
against the oracle, and the workload estimate's argument checks (no GPU: none
of these calls reaches the device)."""
import ctypes

import numpy as np
import pytest

from oracle import dlb as odlb


@pytest.fixture(scope="module")
def gh():
    from paper_2403_17092_amd import gnnhip
    gnnhip.lib()
    return gnnhip


def _cases():
    g = np.random.Generator(np.random.PCG64(17))
    out = [([10, 9, 8, 1, 1, 1], [1, 1]), ([1] * 9, [1, 2]), ([5, 5, 5, 5], [0, 1, 1]),
           ([], [1, 1]), ([0, 0, 3], [1]), ([7], [0.2, 0.3, 0.5])]
    for _ in range(40):
        n, k = int(g.integers(0, 200)), int(g.integers(1, 9))
        if g.random() < 0.5:
            work = g.integers(0, 10**6, n)
        else:  # skewed, with ties
            work = (g.pareto(1.2, n) * 1000).astype(np.int64) // 7 * 7
        ratio = g.random(k) * (g.random(k) > 0.2) + 1e-3
        out.append((work.tolist(), ratio.tolist()))
    return out


def test_assign_matches_the_oracle(gh):
    for work, ratio in _cases():
        w_c, l_c = gh.dlb_assign(work, ratio)
        w_o, l_o = odlb.assign(work, ratio)
        assert w_c == w_o.tolist(), (work, ratio)
        assert l_c == l_o.tolist()


def test_ratio_matches_the_oracle(gh):
    g = np.random.Generator(np.random.PCG64(3))
    cases = [([100, 300], [1.0, 2.0], [0.5, 0.5], 0.05), ([100, 300], [1.0, 1.0], [0.5, 0.5], 0.0),
             ([0, 100, 200], [0.0, 1.0, 4.0], [0.5, 0.25, 0.25], 0.0), ([0, 0], [0, 0], [2, 6], 0.1)]
    for _ in range(30):
        k = int(g.integers(1, 6))
        load = (g.integers(0, 10**7, k) * (g.random(k) > 0.15)).tolist()
        sec = (g.random(k) * 3).tolist()
        prev = (g.random(k) + 0.01).tolist()
        cases.append((load, sec, prev, float(g.choice([0.0, 0.02, 0.3]))))
    for load, sec, prev, tol in cases:
        got = gh.dlb_ratio(load, sec, prev, tol)
        want = odlb.update_ratio(load, sec, prev, tol)
        np.testing.assert_allclose(got, want, rtol=1e-15, atol=0)
        assert abs(sum(got) - 1.0) < 1e-12


def test_bad_arguments_are_rejected(gh):
    L = gh.lib()
    i64a = (ctypes.c_int64 * 2)(5, -1)
    r = (ctypes.c_double * 2)(1.0, 1.0)
    out = (ctypes.c_int32 * 2)()
    assert L.gnn_dlb_assign(i64a, 2, r, 2, out, None) == gh.EINVAL          # negative work
    ok = (ctypes.c_int64 * 2)(5, 1)
    zero = (ctypes.c_double * 2)(0.0, 0.0)
    assert L.gnn_dlb_assign(ok, 2, zero, 2, out, None) == gh.EINVAL          # ratios sum to 0
    assert L.gnn_dlb_assign(ok, 2, r, 0, out, None) == gh.EINVAL             # no worker
    nan = (ctypes.c_double * 2)(float("nan"), 1.0)
    assert L.gnn_dlb_assign(ok, 2, nan, 2, out, None) == gh.EINVAL
    sec = (ctypes.c_double * 2)(1.0, 1.0)
    res = (ctypes.c_double * 2)()
    assert L.gnn_dlb_ratio(ok, sec, zero, 2, 0.0, res) == gh.EINVAL          # prev sums to 0
    assert L.gnn_dlb_ratio(ok, sec, r, 2, -1.0, res) == gh.EINVAL            # tolerance < 0
    assert L.gnn_dlb_ratio(i64a, sec, r, 2, 0.0, res) == gh.EINVAL           # negative load


def test_estimate_rejects_bad_arguments_before_any_launch(gh):
    L = gh.lib()
    m = gh._model_struct("sage_mean", (8, 8, 4))
    csr = gh.CCsr()
    fan = gh._i32arr([4, 2])
    ids = (ctypes.c_void_p * 1)(None)
    keys = (ctypes.c_uint64 * 1)(1)
    work = ctypes.c_void_p(16)  # never written: every call below fails on the host
    ws = ctypes.c_void_p(16)
    assert L.gnn_estimate_work(None, ctypes.byref(csr), ids, keys, 1, 4, fan, work, None, ws, 1 << 20,
                               None) == gh.EINVAL                           # null model
    assert L.gnn_estimate_work(ctypes.byref(m), ctypes.byref(csr), ids, keys, 1, 4, fan, work, None,
                               ws, 1 << 20, None) == gh.EINVAL              # null CSR arrays
    bad = gh._model_struct("sage_mean", (8, 0, 4))
    assert L.gnn_shadow_estimate_work(ctypes.byref(bad), ctypes.byref(csr), ids, keys, 1, 4, 5, 2,
                                      work, None, ws, 1 << 20, None) == gh.EINVAL
    assert L.gnn_estimate_workspace_bytes(4, fan, 2, 1000) > 0
    assert L.gnn_estimate_workspace_bytes(4, fan, 9, 1000) == 0             # layer count out of range
    assert L.gnn_shadow_estimate_workspace_bytes(4, 5, 2) > L.gnn_shadow_workspace_bytes(4, 5, 2)
    assert L.gnn_shadow_estimate_workspace_bytes(4, 5, 7) == 0
