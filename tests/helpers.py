"""Small hand-made graphs and comparison helpers shared by the tests."""
from __future__ import annotations

import numpy as np


def csr_from_edges(n, edges):
    """Simple undirected CSR (int64 rowptr, int32 col) from an edge list."""
    adj = [set() for _ in range(n)]
    for u, v in edges:
        if u != v:
            adj[u].add(v)
            adj[v].add(u)
    rowptr = np.zeros(n + 1, np.int64)
    for i in range(n):
        rowptr[i + 1] = rowptr[i] + len(adj[i])
    col = np.array([w for i in range(n) for w in sorted(adj[i])], np.int32)
    return rowptr, col


def path_graph(n):
    return csr_from_edges(n, [(i, i + 1) for i in range(n - 1)])


def star_graph(leaves):
    return csr_from_edges(leaves + 1, [(0, i) for i in range(1, leaves + 1)])


def complete_graph(n):
    return csr_from_edges(n, [(i, j) for i in range(n) for j in range(i + 1, n)])


def cycle_graph(n):
    return csr_from_edges(n, [(i, (i + 1) % n) for i in range(n)])


def mixed_graph():
    """Hub 0 with 40 leaves, a K5 on 41..45, a path 46..50 and an isolated node 51."""
    e = [(0, i) for i in range(1, 41)]
    e += [(i, j) for i in range(41, 46) for j in range(i + 1, 46)]
    e += [(i, i + 1) for i in range(46, 50)]
    e += [(3, 41), (7, 46)]
    return csr_from_edges(52, e)


def random_graph(n, p, seed):
    g = np.random.Generator(np.random.PCG64(seed))
    m = g.random((n, n)) < p
    edges = [(i, j) for i in range(n) for j in range(i + 1, n) if m[i, j]]
    return csr_from_edges(n, edges)


def dense_adjacency(rowptr, col):
    n = rowptr.shape[0] - 1
    A = np.zeros((n, n))
    for v in range(n):
        A[v, col[rowptr[v]:rowptr[v + 1]]] = 1.0
    return A


def rel_err(x, y):
    """Normwise relative error ||x - y|| / ||y|| (0 when both are empty or zero)."""
    x = np.asarray(x, np.float64)
    y = np.asarray(y, np.float64)
    d = np.linalg.norm((x - y).ravel())
    n = np.linalg.norm(y.ravel())
    return d / n if n > 0 else d


def assert_close(x, y, tol, what=""):
    """Normwise relative error ||x - y|| / ||y|| <= tol (the stated relative
    tolerance), plus an elementwise guard |x - y| <= 8 tol (|y| + rms(y)):
    an element produced by cancellation carries the rounding error of its
    summed terms, whose scale is the tensor's root-mean-square, not |y|."""
    x = np.asarray(x, np.float64)
    y = np.asarray(y, np.float64)
    assert x.shape == y.shape, (what, x.shape, y.shape)
    if y.size == 0:
        return
    e = rel_err(x, y)
    assert e <= tol, f"{what}: normwise relative error {e:.3e} > {tol:.1e}"
    scale = np.abs(y) + np.sqrt(np.mean(y * y))
    ratio = np.abs(x - y) / (8 * tol * scale + 1e-30)
    nbad = int((ratio > 1).sum())
    assert nbad == 0, (
        f"{what}: {nbad} of {y.size} elements outside the elementwise guard "
        f"(worst {ratio.max():.2f}x, normwise {e:.2e})")
