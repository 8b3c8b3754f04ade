"""Seeded synthetic graphs shaped like the paper's workloads.

The paper trains on Reddit, ogbn-products and MAG240M (Table 2).  None of them
is available here, so power-law stand-ins are generated instead:

* Chung-Lu with a power-law expected-degree sequence (exponent gamma);
* R-MAT with quadrant probabilities (a, b, c, d).

Both are symmetrised, stripped of self loops and duplicate edges, relabelled
through a random vertex permutation and returned as CSR (rows sorted
ascending).  This module holds no arithmetic of the training method.
"""
from __future__ import annotations

import ctypes
import math
import os
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libwlgen.so")
_lib = None


def build_generator(force: bool = False) -> str:
    """Compile the host generator (g++ + OpenMP) next to this file."""
    src = os.path.join(_HERE, "gen.cpp")
    if force or not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(src):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        subprocess.check_call(["g++", "-O3", "-fopenmp", "-shared", "-fPIC", "-std=c++17", src, "-o", tmp])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _gen():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build_generator()
        lib = ctypes.CDLL(_LIB_PATH)
        P = ctypes.c_void_p
        i64, i32, u64, f64 = ctypes.c_int64, ctypes.c_int32, ctypes.c_uint64, ctypes.c_double
        lib.wl_rmat_pairs.argtypes = [i64, i32, i64, f64, f64, f64, u64, P, P]
        lib.wl_chunglu_pairs.argtypes = [i64, P, i64, u64, P, P]
        lib.wl_permute_pairs.argtypes = [i64, P, P, P]
        lib.wl_count_degrees.argtypes = [i64, P, P, P]
        lib.wl_scatter_pairs.argtypes = [i64, P, P, P, P]
        lib.wl_sort_unique_rows.argtypes = [i64, P, P, P]
        lib.wl_compact_rows.argtypes = [i64, P, P, P, P]
        lib.wl_normal_rows_f32.argtypes = [i64, i64, i32, i64, u64, P]
        lib.wl_normal_rows_bf16.argtypes = [i64, i64, i32, i64, u64, P]
        lib.wl_num_threads.restype = i32
        _lib = lib
    return _lib


def _p(a: np.ndarray) -> int:
    return a.ctypes.data


@dataclass
class CSRGraph:
    """Simple undirected graph in CSR form: neighbours of v are col[rowptr[v]:rowptr[v+1]],
    ascending, no self loops, no duplicates, and (u in N(v)) == (v in N(u))."""
    rowptr: np.ndarray  # int64 [N+1]
    col: np.ndarray     # int32 [E]

    @property
    def num_nodes(self) -> int:
        return int(self.rowptr.shape[0] - 1)

    @property
    def num_edges(self) -> int:
        return int(self.col.shape[0])

    def degrees(self) -> np.ndarray:
        return np.diff(self.rowptr)


def _quiet(msg: str) -> None:
    pass


def pairs_to_csr(n: int, src: np.ndarray, dst: np.ndarray, log=_quiet) -> CSRGraph:
    """Symmetrise, drop self loops and rejected (-1) pairs, sort rows, dedup.
    `log` receives one line per finished stage."""
    return _pairs_to_csr(n, [src, dst], log)


def _pairs_to_csr(n: int, pairs: list, log=_quiet) -> CSRGraph:
    """pairs_to_csr on pairs = [src, dst]; the list is emptied once the pairs are
    scattered into rows, so a caller that keeps no other reference frees them
    before the sort (lower peak memory for the largest graphs)."""
    lib = _gen()
    src, dst = pairs
    m = int(src.shape[0])
    deg = np.zeros(n + 1, dtype=np.int64)
    lib.wl_count_degrees(m, _p(src), _p(dst), _p(deg))
    tmp_ptr = np.zeros(n + 1, dtype=np.int64)
    np.cumsum(deg[:n], out=tmp_ptr[1:])
    del deg
    cursor = tmp_ptr[:n].copy()
    tmp_col = np.empty(int(tmp_ptr[n]), dtype=np.int32)
    lib.wl_scatter_pairs(m, _p(src), _p(dst), _p(cursor), _p(tmp_col))
    del cursor, src, dst
    pairs.clear()
    log(f"scattered {tmp_col.shape[0]} directed pairs")
    newdeg = np.empty(n, dtype=np.int64)
    lib.wl_sort_unique_rows(n, _p(tmp_ptr), _p(tmp_col), _p(newdeg))
    log("sorted and deduplicated rows")
    rowptr = np.zeros(n + 1, dtype=np.int64)
    np.cumsum(newdeg, out=rowptr[1:])
    del newdeg
    col = np.empty(int(rowptr[n]), dtype=np.int32)
    lib.wl_compact_rows(n, _p(tmp_ptr), _p(tmp_col), _p(rowptr), _p(col))
    return CSRGraph(rowptr=rowptr, col=col)


def _permutation(n: int, seed: int) -> np.ndarray:
    return np.random.Generator(np.random.PCG64([seed, 0xBEEF])).permutation(n).astype(np.int32)


def rmat_graph(n: int, n_pairs: int, seed: int, a=0.57, b=0.19, c=0.19, log=_quiet) -> CSRGraph:
    """R-MAT on 2**ceil(log2 n) ids; pairs landing at ids >= n are rejected."""
    lib = _gen()
    scale = max(1, int(math.ceil(math.log2(n))))
    src = np.empty(n_pairs, dtype=np.int32)
    dst = np.empty(n_pairs, dtype=np.int32)
    lib.wl_rmat_pairs(n_pairs, scale, n, a, b, c, seed, _p(src), _p(dst))
    perm = _permutation(n, seed)
    lib.wl_permute_pairs(n_pairs, _p(perm), _p(src), _p(dst))
    del perm
    log(f"drew {n_pairs} R-MAT pairs")
    pairs = [src, dst]
    del src, dst
    return _pairs_to_csr(n, pairs, log)


def chunglu_weights(n: int, avg_degree: float, gamma: float) -> np.ndarray:
    """Expected degrees w_i = c (i + i0)^(-1/(gamma-1)) with mean avg_degree and the
    largest weight equal to sqrt(sum w) (the usual cap that keeps w_i w_j / sum w <= 1)."""
    alpha = 1.0 / (gamma - 1.0)
    idx = np.arange(n, dtype=np.float64)
    total = n * avg_degree

    def wmax_excess(i0: float) -> float:
        shape = (idx + i0) ** (-alpha)
        c = total / shape.sum()
        return c * i0 ** (-alpha) - math.sqrt(total)

    lo, hi = 1e-6, float(n)
    for _ in range(200):  # bisection on log scale: wmax decreases as i0 grows
        mid = math.sqrt(lo * hi)
        if wmax_excess(mid) > 0:
            lo = mid
        else:
            hi = mid
    i0 = math.sqrt(lo * hi)
    shape = (idx + i0) ** (-alpha)
    return shape * (total / shape.sum())


def chunglu_graph(n: int, avg_degree: float, gamma: float, seed: int, oversample: float = 1.0,
                  log=_quiet) -> CSRGraph:
    lib = _gen()
    w = chunglu_weights(n, avg_degree, gamma)
    cdf = np.cumsum(w)
    cdf /= cdf[-1]
    cdf[-1] = 1.0
    n_pairs = int(round(n * avg_degree / 2.0 * oversample))
    src = np.empty(n_pairs, dtype=np.int32)
    dst = np.empty(n_pairs, dtype=np.int32)
    lib.wl_chunglu_pairs(n_pairs, _p(cdf), n, seed, _p(src), _p(dst))
    perm = _permutation(n, seed)
    lib.wl_permute_pairs(n_pairs, _p(perm), _p(src), _p(dst))
    del perm
    log(f"drew {n_pairs} Chung-Lu pairs")
    pairs = [src, dst]
    del src, dst
    return _pairs_to_csr(n, pairs, log)


def normal_features(n: int, f: int, seed: int, dtype: str = "f32", stride: int | None = None,
                    row_lo: int = 0, row_hi: int | None = None) -> np.ndarray:
    """N(0,1) rows [row_lo, row_hi) as a [rows x stride] array (float32, or uint16
    holding bfloat16 bits rounded to nearest even).  Row r depends only on (seed, r)."""
    lib = _gen()
    stride = f if stride is None else stride
    row_hi = n if row_hi is None else row_hi
    rows = row_hi - row_lo
    if dtype == "f32":
        out = np.zeros((rows, stride), dtype=np.float32)
        lib.wl_normal_rows_f32(row_lo, row_hi, f, stride, seed, _p(out))
    elif dtype == "bf16":
        out = np.zeros((rows, stride), dtype=np.uint16)
        lib.wl_normal_rows_bf16(row_lo, row_hi, f, stride, seed, _p(out))
    else:
        raise ValueError(dtype)
    return out
