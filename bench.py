"""Throughput of one sampling-based GNN training step on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config 5] [--extra 2]
    python bench.py --config 5 --traffic      # counters (rocprofv3), see below

Workload (default, configuration 5, the largest that fits one GPU): 3-layer
GraphSAGE-mean 128-256-256-172 on an R-MAT graph (a, b, c, d = 0.57, 0.19,
0.19, 0.05) of 111M nodes and ~3.33B directed edges (int64 row pointers),
bf16 N(0,1) features of width 128, fanouts [15, 10, 5], 1024 seeds per
batch, SGD lr 0.01; batch s uses sampling key 1 + s.  A step is the whole
path: sampling and relabelling of every hop, the feature fetch (inside the
layer-1 aggregation), forward, loss, backward, SGD, all inside the timed
region with every input resident in HBM.  --extra adds the compact figures
of other workloads (default: configuration 2, the 2.45M-node GraphSAGE).

Prints one JSON line: mini-batches/s, sampled edges/s, per-stage times, the
roofline of the dominant kernel launch (algorithmic and, from the committed
counters, measured), the gather + aggregation bandwidth and the CPU oracle
baseline.

Throughput: the K timed steps run twice, first serially (each step's sampling
and model pass one after the other on one stream: value_serial), then
pipelined (batch i + 1 sampled on a second stream while batch i trains, the
two block slots of the workspace alternating: value_pipelined).  `value` is
the pipelined figure (--serial reports the serial one).  Both time whole
steps with every input resident in HBM.

Dominant kernel: a few untimed steps run with every launch carrying a pair of
HIP events that take the kernel's start and end timestamps (gnn_trace_begin);
the launch with the longest mean duration is the dominant one.  The K timed
steps run with no events at all (they give the throughput); then the same K
steps run again with the stage events and the timestamp events of the
dominant kernel's launches (on the stream they run on), and its mean duration
there divides the launch's algorithmic bytes (HBM-bound kernels) or flops
(GEMMs).

--traffic runs the same workload three times under `rocprofv3 --pmc`
(FETCH_SIZE; WRITE_SIZE; the matrix-instruction counters), each followed by
probes of known size: a plain 256 MiB elementwise copy (the scale from
counter units to bytes) and a 4096^3 library GEMM in fp32 and in bf16 (flops
per matrix-operation count).  It writes every launch's HBM bytes and MFMA
counts to --traffic-out.  A default run reads profiles/traffic.json and
reports, for each launch whose kernel source is unchanged since, the
counter-based fraction of HBM peak (counter_frac) and of MFMA peak (mfma_util)
beside the algorithmic one.  Algorithmic bytes count each distinct row once
(the compulsory traffic), so neither fraction can exceed 1.
"""
from __future__ import annotations

import argparse
import ctypes
import hashlib
import json
import os
import platform
import shutil
import sqlite3
import subprocess
import sys
import tempfile
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0      # MI355X HBM3E, AMD datasheet
FP32_MFMA_TFLOPS = 157.3   # MI355X dense fp32 matrix
MFMA_PEAK_TFLOPS = {"f32": FP32_MFMA_TFLOPS, "bf16": 2500.0}  # dense, per operand type
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")
COPY_PROBE_FLOATS = 64 << 20  # 256 MiB read + 256 MiB written

# source files of each traced kernel (a traffic entry is valid for their hash)
_CSRC = os.path.join(ROOT, "paper_2403_17092_amd", "csrc")
# (the GEMM and gather launches also hash train.hip, which picks their operand
# layouts: a masked or an unmasked instance, a masked gather output)
KERNEL_SOURCES = {
    "begin": ["sample.hip"], "sample": ["sample.hip", "sampler.hpp", "philox.hpp", "relabel.hpp"],
    "scans": ["sample.hip"], "indices": ["sample.hip", "relabel.hpp"],
    "shadow_build": ["shadow.hip", "sampler.hpp", "philox.hpp"], "shadow_scan": ["shadow.hip"],
    "shadow_emit": ["shadow.hip"], "gather": ["gather.hip"],
    "aggregate": ["aggregate.hip", "relabel.hpp"],
    "scatter": ["aggregate.hip", "train.hip"], "relu_mask": ["aggregate.hip"],
    "gemm_fwd": ["gemm.hip", "train.hip"], "gemm_dw": ["gemm.hip", "train.hip"],
    "gemm_dx": ["gemm.hip", "train.hip"], "gemm_bwd": ["gemm.hip", "train.hip"],
    "softmax_xent": ["loss.hip"], "sgd": ["loss.hip"], "fill": ["common.hip"],
    "head": ["head.hip"],
    "gat_scores": ["gat.hip"], "gat_attend": ["gat.hip"], "gat_attend_bwd": ["gat.hip"],
    "gat_score_grad": ["gat.hip"], "gat_colsum": ["gat.hip"], "gat_colsum_final": ["gat.hip"],
    "work": ["dlb.hip"],
}


def _log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def kernel_source_hash(name: str, cfg=None) -> str:
    """Hash of the sources a traced launch runs; a bf16-feature GraphSAGE/GCN
    workload's layer-1 products also run the thin kernels of gemm_thin.hip."""
    files = list(KERNEL_SOURCES.get(name, []))
    if name in ("gemm_fwd", "gemm_dw") and cfg is not None:
        from workloads import configs
        spec = configs.CONFIGS[cfg]
        if spec.feat_dtype == "bf16" and spec.kind in ("sage_mean", "gcn"):
            files.append("gemm_thin.hip")
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(_CSRC, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


class HipEvents:
    """hipEvent_t handles from the HIP runtime already loaded by torch."""

    def __init__(self, n):
        self.rt = ctypes.CDLL("libamdhip64.so.7")
        self.rt.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.rt.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                                ctypes.c_void_p]
        self.rt.hipEventDestroy.argtypes = [ctypes.c_void_p]
        self.ev = []
        for _ in range(n):
            h = ctypes.c_void_p()
            rc = self.rt.hipEventCreate(ctypes.byref(h))
            assert rc == 0, rc
            self.ev.append(h.value)

    def elapsed_ms(self, a, b):
        ms = ctypes.c_float()
        rc = self.rt.hipEventElapsedTime(ctypes.byref(ms), ctypes.c_void_p(self.ev[a]),
                                         ctypes.c_void_p(self.ev[b]))
        assert rc == 0, rc
        return ms.value

    def close(self):
        for e in self.ev:
            self.rt.hipEventDestroy(ctypes.c_void_p(e))


# ---------------------------------------------------------------------------
# launch bookkeeping
# ---------------------------------------------------------------------------
def launch_keys(names):
    """'name#k' for the k-th launch of `name` within one step."""
    seen, keys = {}, []
    for n in names:
        k = seen.get(n, 0)
        seen[n] = k + 1
        keys.append(f"{n}#{k}")
    return keys


SHADOW_HUB_DEGREE = 1024  # the extraction's default (gnn_csr hub_degree 0)


def shadow_row_words(deg, nodes, comp_ptr, B):
    """CSR words the ShaDow extraction must read for one batch: the whole rows
    of the subgraph nodes of degree <= the hub degree, plus one binary search
    (ceil(log2 d) + 1 words of the shorter row) per pair of higher-degree nodes
    of a component."""
    import numpy as np
    d = deg[nodes].astype(np.int64)
    words = float(d[d <= SHADOW_HUB_DEGREE].sum())
    for r in range(B):
        comp = np.concatenate([[r], np.arange(comp_ptr[r], comp_ptr[r + 1])])
        hubs = np.sort(d[comp][d[comp] > SHADOW_HUB_DEGREE])
        for i in range(len(hubs)):  # pair (i, j > i): search in the shorter row hubs[i]
            words += (len(hubs) - 1 - i) * (np.ceil(np.log2(hubs[i])) + 1)
    return words


def gat_launch_model(spec, name, k, layer_block, sz):
    """Algorithmic work of a GAT step's launches (see launch_models); None for
    the launches the models share (sampling, loss, update)."""
    L = len(spec.dims) - 1
    esz0 = 2 if spec.feat_dtype == "bf16" else 4

    def dims(l):
        nd, ns, e = layer_block(l)
        return nd, ns, e, spec.dims[l - 1], spec.dims[l]

    if name == "gather":
        ns = layer_block(1)[1]
        F0 = spec.dims[0]
        return ("hbm", ns * (F0 * esz0 + F0 * 4 + 4),
                f"{ns:.0f} input rows of {F0} x {esz0} B read, written as fp32, ids")
    if name == "gemm_fwd":
        nd, ns, e, fi, fo = dims(k + 1)
        return ("mfma", 2.0 * ns * fi * fo, f"layer {k + 1}: T = H W, 2 x {ns:.0f} x {fi} x {fo} flops")
    if name == "gat_scores":
        nd, ns, e, fi, fo = dims(k + 1)
        return ("hbm", ns * (fo * 4 + 8), f"layer {k + 1}: {ns:.0f} rows of T read, 2 scores written")
    # row reads below count every distinct row once (repeats are cache hits)
    if name == "gat_attend":
        if k == L:  # layer 1's backward: the attention-weighted input rows G
            nd, ns, e, fi, fo = dims(1)
            r, u = e + nd, min(ns, e + nd)
            return ("hbm", u * fi * 4 + r * 8 + nd * (fi * 4 + 16),
                    f"layer 1 backward: {u:.0f} distinct input rows ({fi} x 4 B), scores and ids of "
                    f"{r:.0f} edges, {nd:.0f} rows of G")
        nd, ns, e, fi, fo = dims(k + 1)
        r, u = e + nd, min(ns, e + nd)
        return ("hbm", u * fo * 4 + r * 8 + nd * (fo * 4 + 16),
                f"layer {k + 1}: {u:.0f} distinct rows of T ({fo} x 4 B), scores and ids of {r:.0f} "
                f"edges, {nd:.0f} output rows")
    if name == "gat_attend_bwd":
        l = L - k
        nd, ns, e, fi, fo = dims(l)
        r, u = e + nd, min(ns, e + nd)
        if l == 1:  # no dT: layer 1's weight gradient is formed from G
            return ("hbm", u * fo * 4 + r * 16 + nd * fo * 8,
                    f"layer 1: {u:.0f} distinct rows of T read, scores, ids and two score-gradient "
                    f"adds of {r:.0f} edges; {nd:.0f} output-gradient rows (and mask)")
        return ("hbm", u * fo * 12 + r * 16 + nd * fo * 8,
                f"layer {l}: {u:.0f} distinct rows of T read and of dT added to, scores, ids and two "
                f"score-gradient adds of {r:.0f} edges; {nd:.0f} output-gradient rows (and mask)")
    if name == "gat_score_grad":
        l = L - k
        nd, ns, e, fi, fo = dims(l)
        return ("hbm", ns * (fo * 8 + 8), f"layer {l}: {ns:.0f} rows of dT updated from 2 scores")
    if name == "gemm_dw":
        if k >= L - 1:  # layer 1: dW = G^T dOut, then dW += hh [a_l; a_r]
            nd, ns, e, fi, fo = dims(1)
            f, what = [(2.0 * nd * fi * fo, "G^T dOut"), (2.0 * fi * 2 * fo, "hh a")][k - (L - 1)]
            return ("mfma", f, f"layer 1: {what}, {f:.3g} flops")
        l = L - k
        nd, ns, e, fi, fo = dims(l)
        return ("mfma", 2.0 * ns * fi * fo, f"layer {l}: dW = H^T dT, 2 x {ns:.0f} x {fi} x {fo} flops")
    if name == "gat_colsum":
        # [ds_l | ds_r]^T T per layer (da); layer 1 also H^T [ds_l | ds_r]
        if k == L:
            nd, ns, e, fi, fo = dims(1)
            return ("hbm", ns * (fi * 4 + 8) + 256 * 2048,
                    f"layer 1: {ns:.0f} input rows of {fi} x 4 B and 2 scores read, 256 parts written")
        l = L - k
        nd, ns, e, fi, fo = dims(l)
        return ("hbm", ns * (fo * 4 + 8) + 256 * 2048,
                f"layer {l}: {ns:.0f} rows of T ({fo} x 4 B) and 2 scores read, 256 parts written")
    if name == "gat_colsum_final":
        return ("hbm", 256 * 2048, "256 parts of 2 x 256 column sums read")
    if name == "gemm_dx":
        l = L - k
        nd, ns, e, fi, fo = dims(l)
        return ("mfma", 2.0 * ns * fo * fi, f"layer {l}: dH = dT W^T, 2 x {ns:.0f} x {fo} x {fi} flops")
    if name == "sgd":
        P = sum((a + 2) * b for a, b in zip(spec.dims[:-1], spec.dims[1:]))
        return ("hbm", P * 12, f"{P} weights and gradients")
    return None


# bf16-feature GraphSAGE and GCN runs take layer 1's products on the bf16 MFMA
LAYER1_BF16_MFMA = True


def gemm_layer(spec, key):
    """Layer of a GEMM launch of a GraphSAGE or GCN step: gemm_fwd#k is layer
    k + 1; gemm_bwd#k (a hidden layer's weight and input gradients in one
    launch) counts down from the top layer the backward GEMMs start at; the
    lone gemm_dw is layer 1's (it has no input gradient)."""
    name, k = key.split("#")
    k = int(k)
    L = len(spec.dims) - 1
    head = L >= 2 and spec.dims[-1] <= 64
    top = L - 1 if head else L
    if name == "gemm_fwd":
        return k + 1
    if name == "gemm_bwd":
        return top - k
    if name == "gemm_dw":
        return 1
    return None


def mfma_dtype(spec, key):
    """Operand type of a GEMM launch's matrix instructions."""
    if (LAYER1_BF16_MFMA and spec.feat_dtype == "bf16" and spec.kind in ("sage_mean", "gcn")
            and key.split("#")[0] in ("gemm_fwd", "gemm_dw") and gemm_layer(spec, key) == 1):
        return "bf16"
    return "f32"


def step_dtype(spec):
    """Arithmetic types of a step, for the result line."""
    if spec.feat_dtype == "f32":
        return "f32"
    if LAYER1_BF16_MFMA and spec.kind in ("sage_mean", "gcn"):
        return "bf16 features and layer-1 products / f32"
    return "bf16-features/f32"


def launch_models(spec, keys, sz):
    """Algorithmic work of each launch of one step: key -> (bound, amount, what).

    sz: mean sizes of the timed steps.  Neighbour sampling: sz["hops"][h] =
    (n_dst, n_src, E) of hop h + 1.  ShaDow: sz["union"] = (n, E), sz["root_e"]
    (edges of the root rows), sz["row_elems"] (summed CSR degree of the union's
    nodes).  bound "hbm": amount in bytes; "mfma": amount in flops."""
    L = len(spec.dims) - 1
    F0 = spec.feat_dim
    esz0 = 2 if spec.feat_dtype == "bf16" else 4
    rpb = 8 if spec.rowptr64 else 4
    sage = spec.kind == "sage_mean"
    gin = spec.kind == "gin"
    B = spec.batch

    def layer_block(l):  # (n_dst, n_src, E) of the block layer l runs on
        if spec.shadow:
            n, e = sz["union"]
            return (B, n, sz["root_e"]) if l == L else (n, n, e)
        return sz["hops"][L - l]

    # the output layer and the loss run fused (one "head" launch) when the
    # model has at most 64 classes and two or more layers; the backward GEMM
    # launches then start at layer L - 1
    head = not gin and L >= 2 and spec.dims[-1] <= 64
    top = L - 1 if head else L
    layered = {"aggregate": lambda k: k + 1, "gemm_fwd": lambda k: k + 1,
               "gemm_dw": lambda k: 1, "gemm_bwd": lambda k: top - k, "scatter": lambda k: L - k,
               "relu_mask": lambda k: L - k}
    if gin:
        # two products per layer forward (agg W_a, M W_b); backward, layer L
        # down to 1: dW_b, dM, dW_a, then dAgg (not on layer 1)
        layered.update({"gemm_fwd": lambda k: k // 2 + 1, "gemm_dw": lambda k: L - k // 2,
                        "gemm_dx": lambda k: L - k // 2})
    out = {}
    gemm_io = {}
    for key in keys:
        name, k = key.split("#")
        k = int(k)
        m = None
        if spec.kind == "gat":
            m = gat_launch_model(spec, name, k, layer_block, sz)
            if m is not None:
                out[key] = m
                continue
        if name == "gather":
            n_out = sz["union"][0] if spec.shadow else sz["hops"][-1][1]
            b = n_out * (2 * F0 * esz0 + 4)
            what = f"{n_out:.0f} rows x {F0} x {esz0} B read and written, plus ids"
            if not spec.shadow:  # the launch also compacts the last hop's edges
                nd, _, e = sz["hops"][-1]
                b += e * 16 + nd * 8
                what += f"; {e:.0f} edges compacted"
            m = ("hbm", b, what)
        elif name in layered:
            l = layered[name](k)
            nd, ns, e = layer_block(l)
            fi, fo = spec.dims[l - 1], spec.dims[l]
            esz = esz0 if l == 1 else 4
            xw = 2 * fi if sage else fi
            if gin:
                xw = fi  # the aggregation writes agg; M is the first product's output
            if name == "aggregate":
                # every distinct input row once (the src rows: the dst rows and
                # the rows their edges reach; repeats are cache hits, not HBM)
                rows = min(ns, e + nd)
                b = rows * fi * esz + nd * xw * 4 + 4 * (e + nd + 1) + \
                    (4 * rows if spec.kind == "gcn" else 0)
                what = (f"layer {l}: {rows:.0f} distinct input rows of {fi} x {esz} B "
                        f"({e + nd:.0f} row reads), {nd:.0f} output rows of {xw} x 4 B, indices")
                if l == 1:  # rows of the feature table through the src node ids
                    b += 4 * rows
                    what += ", feature-table row ids"
                    if sage and not spec.shadow:  # the launch also compacts the hop's edges
                        b += e * 16 + nd * 8
                        what += f"; {e:.0f} edges compacted"
                m = ("hbm", b, what)
            elif name.startswith("gemm") and gin:
                # even launches of gemm_fwd are agg W_a (k = fi); of gemm_dw and
                # gemm_dx the W_b products (dW_b, dM: k = fo)
                second = (k % 2 == 1) if name == "gemm_fwd" else (k % 2 == 0)
                kk = fo if second else fi
                m = ("mfma", 2.0 * nd * kk * fo, f"layer {l}: 2 x {nd:.0f} x {kk} x {fo} flops")
            elif name == "gemm_bwd":
                # dW = X^T dZ and dX = dZ W^T of one hidden layer, one launch
                m = ("mfma", 2 * 2.0 * nd * xw * fo,
                     f"layer {l}: dW and dX, 2 x (2 x {nd:.0f} x {xw} x {fo}) flops")
                masked = l < L
                gemm_io[key] = (nd * xw * 4 + nd * fo * (8 if masked else 4) + xw * fo * 4) + \
                               (nd * fo * (8 if masked else 4) + xw * fo * 4 + nd * xw * 4)
            elif name.startswith("gemm"):
                m = ("mfma", 2.0 * nd * xw * fo, f"layer {l}: 2 x {nd:.0f} x {xw} x {fo} flops")
                # compulsory operand bytes: X (bf16 on a bf16 layer 1), the
                # weights, dZ (bf16 on a bf16 layer 1 below two layers; else
                # fp32 with its ReLU mask on hidden layers), the output once
                x16 = l == 1 and mfma_dtype(spec, "gemm_fwd#0") == "bf16"
                ex = 2 if x16 else 4
                masked = l < L
                if name == "gemm_fwd":
                    io = nd * xw * ex + xw * fo * 4 + nd * fo * 4
                elif name == "gemm_dw":
                    dz = nd * fo * (2 if (x16 and L >= 2) else (8 if masked else 4))
                    io = nd * xw * ex + dz + xw * fo * 4
                else:
                    io = nd * fo * (8 if masked else 4) + xw * fo * 4 + nd * xw * 4
                gemm_io[key] = io
            elif name == "scatter" and spec.shadow:
                # atomic adds into every distinct target row (read and written
                # once), the dst gradient rows read once
                rows = min(ns, e + nd)
                b = rows * fi * 8 + nd * fi * 4 + 4 * (e + nd + 1)
                m = ("hbm", b, f"layer {l}: {rows:.0f} distinct target rows of {fi} x 4 B read and "
                               f"written ({e + (0 if sage else nd):.0f} row updates), {nd:.0f} "
                               f"gradient rows read, indices")
            elif name == "scatter":  # gather over the block's transpose
                # each dst gradient row read once (the E edges re-read them),
                # every src row written once; SAGE also reads the self path of
                # the dst rows.  Layer 2 of a bf16 run writes layer 1's
                # pre-activation gradient in bf16, masked by H1 (read once)
                to16 = l == 2 and mfma_dtype(spec, "gemm_dw#0") == "bf16"
                out_b = ns * fi * (4 + 2) if to16 else ns * fi * 4
                b = nd * fi * 4 + out_b + (nd * fi * 4 if sage else 0) + 8 * e + 8 * (ns + nd)
                m = ("hbm", b, f"layer {l}: {nd:.0f} dst gradient rows of {fi} x 4 B read "
                               f"({e:.0f} edge reads), {ns:.0f} gradient rows written"
                               + (" as bf16, masked by H1 (read)" if to16 else "") + ", "
                               + ("self path read, " if sage else "") + "lists and offsets")
            elif name == "relu_mask":
                m = ("hbm", ns * fi * 12, f"layer {l}: {ns:.0f} rows x {fi} x 4 B x 3")
        elif name in ("sample", "scans", "indices") and not spec.shadow:
            nd, ns, e = sz["hops"][k]
            f = spec.fanouts[k]
            if name == "sample":
                b = nd * (4 + 2 * rpb + 4 + 4 * f + 8) + e * (4 + 8)
                m = ("hbm", b, f"hop {k + 1}: {nd:.0f} dst (id, row bounds, padded row, count, "
                               f"first-occurrence word) + {e:.0f} picks (column word, word update)")
            elif name == "scans":
                b = nd * (4 + 4 + 4 * f) + e * 8 + 4 * (nd + 1) + ns * 12
                m = ("hbm", b, f"hop {k + 1}: {nd:.0f} x (1 + {f}) positions, {e:.0f} word reads, "
                               f"indptr, {ns:.0f} new ids")
            else:
                b = e * 16 + nd * 8
                m = ("hbm", b, f"hop {k + 1}: {e:.0f} edges (key, local id, index, count)")
        elif name == "shadow_build":
            n, e = sz["union"]
            b = sz["row_elems"] * 4 + n * (2 * rpb + 12) + e * 4
            m = ("hbm", b, f"{sz['row_elems']:.0f} CSR row words (rows of degree <= "
                           f"{SHADOW_HUB_DEGREE} read, higher-degree pairs searched) of the "
                           f"{n:.0f} subgraph nodes, "
                           f"node ids, row counts, {e:.0f} induced edges")
        elif name == "shadow_emit":
            n, e = sz["union"]
            m = ("hbm", e * 8 + n * 16, f"{e:.0f} edges read and written, {n:.0f} rows")
        elif name == "head":
            fi, C = spec.dims[L - 1], spec.dims[L]
            xw = 2 * fi if sage else fi
            m = ("mfma", 3 * 2.0 * B * xw * C,
                 f"output layer: 3 products (Z, dX, dW) of 2 x {B} x {xw} x {C} flops")
        elif name == "softmax_xent":
            m = ("hbm", B * spec.dims[-1] * 8, f"{B} x {spec.dims[-1]} logits read, gradients written")
        elif name == "sgd":
            P = sum((2 * a if sage else (a + b if gin else a)) * b
                    for a, b in zip(spec.dims[:-1], spec.dims[1:]))
            b, what = P * 12, f"{P} weights and gradients"
            if head:
                n_part = -(-B // 16) * spec.dims[L - 1] * (2 if sage else 1) * spec.dims[L]
                b += n_part * 4
                what += f", {n_part} output-layer gradient partials"
            if mfma_dtype(spec, "gemm_dw#0") == "bf16" and L >= 2:
                # layer 1's weight gradient comes as partials over row chunks
                # (at least 512 rows each, a multiple of 8 chunks, at most 32)
                nd1 = layer_block(1)[0]
                chunks = min(32, -(-int(-(-nd1 // 512)) // 8) * 8)
                n_part = chunks * spec.dims[0] * (2 if sage else 1) * spec.dims[1]
                b += n_part * 4
                what += f", {n_part:.0f} layer-1 gradient partials"
            m = ("hbm", b, what)
        if m is not None:
            out[key] = m
    # a product whose operand bytes take longer at HBM peak than its flops at
    # the matrix peak of its operand type is bound by HBM (the roofline's
    # ridge: 19.7 flop/B for fp32, 312 for bf16)
    for key, io in gemm_io.items():
        b, flops, what = out[key]
        peak = MFMA_PEAK_TFLOPS[mfma_dtype(spec, key)] * 1e12
        if io / (HBM_PEAK_GBS * 1e9) > flops / peak:
            out[key] = ("hbm", io, f"{what} at {flops / io:.1f} flop/B, below the "
                                   f"{peak / (HBM_PEAK_GBS * 1e9):.0f} flop/B ridge: {io:.0f} operand "
                                   f"bytes (X, W, dZ and its mask, output once)")
    return out


# ---------------------------------------------------------------------------
# dynamic load balancing (workload estimate and assignment)
# ---------------------------------------------------------------------------
def dlb_leg(gnnhip, torch, spec, csr, batches):
    """Workload estimate of the timed batches (not part of the throughput),
    and how far a 1 : 2 split of them between two workers (a worker twice as
    fast takes two thirds) lands from its targets: by batch count (the first
    third of the batches to the slower worker) and by estimated workload
    (gnn_dlb_assign)."""
    n = len(batches)
    shadow = (spec.shadow_fanout, spec.shadow_hops) if spec.shadow else None

    def estimate():
        return gnnhip.estimate_work(csr, spec.kind, spec.dims, batches, spec.batch,
                                    fanouts=None if shadow else spec.fanouts, shadow=shadow)

    estimate()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    work, _ = estimate()
    torch.cuda.synchronize()
    el = time.perf_counter() - t0
    assert gnnhip.check_errors() == 0
    work = [int(x) for x in work.cpu().tolist()]
    total = sum(work)
    target = [total / 3.0, 2.0 * total / 3.0]
    n0 = int(round(n / 3.0))
    by_count = [sum(work[:n0]), sum(work[n0:])]
    _, by_work = gnnhip.dlb_assign(work, [1.0, 2.0])
    mean = total / max(1, n)
    std = (sum((x - mean) ** 2 for x in work) / max(1, n)) ** 0.5

    def off(loads):
        return max(abs(l - t) / t for l, t in zip(loads, target)) if total else 0.0

    return {"estimate_batches_per_s": n / el, "batches": n, "work_mean": mean,
            "work_cv": std / mean if mean else 0.0,
            "split": "two workers, ratio 1 : 2",
            "off_target_by_count": off(by_count), "off_target_by_workload": off(by_work)}


# ---------------------------------------------------------------------------
# features in host memory, fetched through the GPU feature cache
# ---------------------------------------------------------------------------
def feature_cache_leg(gnnhip, torch, spec, w, csr, labels, seeds, steps, first, nb, dev):
    """Serial training steps with the feature table in pinned host memory
    (read in place by the GPU over the host link): through an LRU cache in HBM
    holding 10% of the rows (warmed first by as many other batches of the
    epoch, as the paper's cache fills over an epoch), and, as the baseline, the plain step
    reading every row it needs in place (zero-copy: the layer-1 aggregation
    reads the host table through the block's node ids)."""
    import numpy as np
    F = spec.feat_dim
    xdt = gnnhip.BF16 if spec.feat_dtype == "bf16" else gnnhip.F32
    feats = w.features.view(np.int16) if spec.feat_dtype == "bf16" else w.features
    t0 = time.perf_counter()
    X_host = torch.as_tensor(feats).pin_memory()
    pin_s = time.perf_counter() - t0
    row_bytes = F * X_host.element_size()
    out = {"features_in": "pinned host memory, read in place by the GPU",
           "row_bytes": row_bytes, "pin_s": round(pin_s, 1)}
    ways = 16
    S = max(1, int(w.graph.num_nodes * 0.10) // ways)
    cache = gnnhip.FeatureCache(S, ways, F, xdt, dev)
    tr = gnnhip.Trainer(spec.kind, spec.dims, w.weights, spec.batch, spec.fanouts,
                        w.graph.num_nodes, xdt, dev, cache_sets=S)
    stats = torch.zeros(2, dtype=torch.int64, device=dev)

    def run_cached(i):
        s = (first + i) % nb
        tr.step_cached(csr, X_host, cache, stats, labels, seeds[s], w.rng_key(s), spec.lr)

    # warm-up pass over as many other batches (later steps of the epoch: fresh
    # seeds and keys), so the timed batches hit what earlier batches left
    from workloads import configs
    base = max(nb, spec.steps)
    for i in range(steps):
        ws_ = torch.as_tensor(configs.make_seeds(w.graph.num_nodes, spec.batch, spec.seed_seed,
                                                 base + i)).to(dev)
        tr.step_cached(csr, X_host, cache, stats, labels, ws_, w.rng_key(base + i), spec.lr)
    torch.cuda.synchronize()
    stats.zero_()
    t0 = time.perf_counter()
    for i in range(steps):
        run_cached(i)
    torch.cuda.synchronize()
    el = time.perf_counter() - t0
    assert gnnhip.check_errors() == 0
    h, m = (int(x) for x in stats.cpu().tolist())
    out["cache"] = {"mini_batches_per_s": steps / el, "cache_rows": S * ways,
                    "cache_fraction_of_rows": S * ways / w.graph.num_nodes,
                    "hit_rate": h / max(1, h + m), "rows_per_step": (h + m) / steps,
                    "host_link_bytes_per_step": m * row_bytes / steps,
                    "host_link_GB_per_s": m * row_bytes / el / 1e9}
    del tr, cache
    # zero-copy baseline: the same serial steps, every feature row read from
    # host memory by the layer-1 aggregation
    tz = gnnhip.Trainer(spec.kind, spec.dims, w.weights, spec.batch, spec.fanouts,
                        w.graph.num_nodes, xdt, dev)

    def run_zero(i):
        s = (first + i) % nb
        tz.step(csr, X_host, labels, seeds[s], w.rng_key(s), spec.lr)

    run_zero(0)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        run_zero(i)
    torch.cuda.synchronize()
    el = time.perf_counter() - t0
    assert gnnhip.check_errors() == 0
    rows = out["cache"]["rows_per_step"]
    out["zero_copy"] = {"mini_batches_per_s": steps / el, "rows_per_step": rows,
                        "host_link_bytes_per_step": rows * row_bytes,
                        "host_link_GB_per_s": rows * row_bytes * steps / el / 1e9}
    out["cache_speedup"] = out["cache"]["mini_batches_per_s"] / out["zero_copy"]["mini_batches_per_s"]
    del tz, X_host
    return out


# ---------------------------------------------------------------------------
# the CPU oracle baseline
# ---------------------------------------------------------------------------
def cpu_baseline(w, seconds: float):
    """The CPU oracle, untouched, timed single-threaded on consecutive steps."""
    from threadpoolctl import threadpool_limits

    from oracle import model as omodel
    from oracle import shadow as oshadow
    spec = w.spec
    W = [x.astype("float64") for x in w.weights]
    done, edges, t0 = 0, 0, time.perf_counter()
    with threadpool_limits(limits=1):
        while True:
            s = done % len(w.seeds)
            if spec.shadow:
                r = oshadow.shadow_train_step(w.graph.rowptr, w.graph.col, w.features, w.labels,
                                              w.seeds[s], spec.shadow_fanout, spec.shadow_hops,
                                              w.rng_key(s), spec.kind, W, spec.lr)
                edges += r["block"].n_edges
            else:
                r = omodel.train_step(w.graph.rowptr, w.graph.col, w.features, w.labels, w.seeds[s],
                                      spec.fanouts, w.rng_key(s), spec.kind, W, spec.lr)
                edges += sum(b.n_edges for b in r["blocks"])
            W = r["W_new"]
            done += 1
            el = time.perf_counter() - t0
            if el >= seconds:
                break
    return done, edges, el


# ---------------------------------------------------------------------------
# counters: rocprofv3 --pmc passes in child processes
# ---------------------------------------------------------------------------
# One pass per counter group (rocprofv3 does not split groups over passes).
# FETCH_SIZE and WRITE_SIZE give the HBM-side bytes of each launch (scaled by
# a plain copy of known size); the MFMA pass gives each launch's matrix
# operations (scaled by a library GEMM of known size) and matrix-core busy
# cycles.
PMC_PASSES = [["FETCH_SIZE"], ["WRITE_SIZE"],
              ["SQ_INSTS_VALU_MFMA_MOPS_F32", "SQ_INSTS_VALU_MFMA_MOPS_BF16", "SQ_VALU_MFMA_BUSY_CYCLES",
               "SQ_BUSY_CYCLES", "GRBM_GUI_ACTIVE"]]
GEMM_PROBE_N = 4096  # the MFMA counters' probe: [N x N] x [N x N] in fp32 and in bf16


def _pmc_pass(counters, cfg, steps, warmup, tmp):
    tag = counters[0]
    d = os.path.join(tmp, tag)
    names_file = os.path.join(tmp, f"names_{tag}.json")
    cmd = ["timeout", "-s", "KILL", "300", "rocprofv3", "--pmc"] + counters + [
        "-d", d, "-o", "run", "--", sys.executable, os.path.join(ROOT, "bench.py"), "--config",
        str(cfg), "--pmc-child", "--steps", str(steps), "--warmup", str(warmup), "--names-out",
        names_file]
    _log("running:", " ".join(cmd))
    r = subprocess.run(cmd, cwd=tmp, stdout=sys.stderr, stderr=sys.stderr)
    db = None
    for root, _, files in os.walk(d):
        if "run_results.db" in files:
            db = os.path.join(root, "run_results.db")
    if db is None or not os.path.exists(names_file):
        raise RuntimeError(f"rocprofv3 pass {counters} failed (rc {r.returncode})")
    with open(names_file) as fh:
        names = json.load(fh)
    con = sqlite3.connect(db)
    per_step = len(names)
    keys = launch_keys(names)
    per_launch, probes = {}, {}
    for counter in counters:
        rows = con.execute("select dispatch_id, kernel_name, value from counters_collection "
                           "where counter_name = ? order by dispatch_id", (counter,)).fetchall()
        gnn = [v for _, k, v in rows if "gnn::" in k]
        last = gnn[-steps * per_step:]
        assert len(last) == steps * per_step, (counter, len(gnn), per_step)
        for i, key in enumerate(keys):
            per_launch.setdefault(key, {})[counter] = sum(last[s * per_step + i]
                                                          for s in range(steps)) / steps
        # the probes run after the steps: the copy, then the fp32 and bf16 GEMMs
        last_gnn = max(i for i, (_, k, _) in enumerate(rows) if "gnn::" in k)
        probes[counter] = [(k, v) for _, k, v in rows[last_gnn + 1:]]
    return per_launch, probes


def _probe_value(probe, pick):
    """Value of the probe dispatch chosen by pick(list of (kernel, value))."""
    return pick(probe) if probe else None


def measure_traffic(args):
    from workloads import configs
    spec = configs.CONFIGS[args.config]
    tmp = tempfile.mkdtemp(prefix="gnn_traffic_")
    fetch, pf = _pmc_pass(PMC_PASSES[0], args.config, args.steps, args.warmup, tmp)
    write, pw = _pmc_pass(PMC_PASSES[1], args.config, args.steps, args.warmup, tmp)
    mfma, pm = {}, {c: [] for c in PMC_PASSES[2]}
    if not args.no_mfma_pass:
        try:
            mfma, pm = _pmc_pass(PMC_PASSES[2], args.config, args.steps, args.warmup, tmp)
        except (RuntimeError, AssertionError, ValueError) as e:  # counters missing on this device
            _log(f"MFMA counter pass failed: {e}")

    def copy_kib(probe):  # the copy: the elementwise multiply after the steps
        return next(v for k, v in probe if "MulFunctor" in k)

    probe_bytes = COPY_PROBE_FLOATS * 4
    fetch_copy, write_copy = copy_kib(pf["FETCH_SIZE"]), copy_kib(pw["WRITE_SIZE"])
    f_scale = probe_bytes / (fetch_copy * 1024.0)  # counter KiB -> bytes
    w_scale = probe_bytes / (write_copy * 1024.0)
    # the GEMM probes: the dispatch with the most matrix operations of each type
    gemm_flops = 2.0 * GEMM_PROBE_N ** 3
    mops = {dt: max((v for _, v in pm[f"SQ_INSTS_VALU_MFMA_MOPS_{c}"]), default=0.0)
            for dt, c in (("f32", "F32"), ("bf16", "BF16"))}
    flops_per_mop = {dt: (gemm_flops / m if m else None) for dt, m in mops.items()}
    entries = {}
    for key in fetch:
        name = key.split("#")[0]
        e = {"fetch_kib": fetch[key]["FETCH_SIZE"], "write_kib": write[key]["WRITE_SIZE"],
             "bytes": fetch[key]["FETCH_SIZE"] * 1024.0 * f_scale
             + write[key]["WRITE_SIZE"] * 1024.0 * w_scale,
             "source": kernel_source_hash(name, args.config)}
        e.update({c.lower(): v for c, v in mfma.get(key, {}).items()})
        entries[f"config{args.config}:{key}"] = e
    result = {"workload": spec.name, "config": args.config,
              "copy_probe": {"bytes_each_way": probe_bytes, "fetch_kib": fetch_copy,
                             "write_kib": write_copy, "fetch_scale": f_scale, "write_scale": w_scale},
              "mfma_probe": {"gemm_n": GEMM_PROBE_N, "flops_each": gemm_flops, "mops": mops,
                             "flops_per_mop": flops_per_mop,
                             "dispatches_after_steps": {c: pm[c] for c in PMC_PASSES[2]}},
              "command": "python bench.py --config %d --traffic --steps %d --warmup %d"
                         % (args.config, args.steps, args.warmup),
              "entries": entries}
    old = {}
    if os.path.exists(args.traffic_out):
        with open(args.traffic_out) as fh:
            old = json.load(fh)
    old.setdefault("runs", {})[f"config{args.config}"] = result
    os.makedirs(os.path.dirname(os.path.abspath(args.traffic_out)), exist_ok=True)
    with open(args.traffic_out, "w") as fh:
        json.dump(old, fh, indent=1, sort_keys=True)
    shutil.rmtree(tmp, ignore_errors=True)
    print(json.dumps(result))


def lookup_counters(cfg, key):
    """The committed counter entry of a launch, if taken from the current source."""
    if not os.path.exists(TRAFFIC_FILE):
        return None
    with open(TRAFFIC_FILE) as fh:
        data = json.load(fh)
    e = data.get("runs", {}).get(f"config{cfg}", {}).get("entries", {}).get(f"config{cfg}:{key}")
    if not e or e.get("source") != kernel_source_hash(key.split("#")[0], cfg):
        return None
    return e


def mfma_flops_per_mop(cfg):
    """Flops per SQ_INSTS_VALU_MFMA_MOPS_* unit from the committed GEMM probe
    (fp32, bf16), or None."""
    if not os.path.exists(TRAFFIC_FILE):
        return None
    with open(TRAFFIC_FILE) as fh:
        data = json.load(fh)
    return data.get("runs", {}).get(f"config{cfg}", {}).get("mfma_probe", {}).get("flops_per_mop")


# ---------------------------------------------------------------------------
def measure(cfg, args, full):
    """Throughput and rooflines of one workload; `full` adds the load-balancer
    estimate, the host-feature leg and the CPU oracle baseline."""
    import numpy as np
    import torch

    from paper_2403_17092_amd import gnnhip
    from workloads import configs

    spec = configs.CONFIGS[cfg]
    t = time.time()
    cal_steps = 3
    nsteps = args.warmup + cal_steps + args.steps
    w = configs.make_workload(spec, steps=min(spec.steps, nsteps) if spec.steps > 1 else 1,
                              log=lambda m: _log(f"{spec.name}: {m}"))
    gen_s = time.time() - t
    _log(f"workload {spec.name}: {w.graph.num_nodes} nodes, {w.graph.num_edges} edges "
         f"({gen_s:.1f} s)")
    dev = torch.device("cuda:0")
    t = time.time()
    rp = w.graph.rowptr if spec.rowptr64 else w.graph.rowptr.astype(np.int32)
    csr = gnnhip.Csr(torch.as_tensor(rp).to(dev), torch.as_tensor(w.graph.col).to(dev))
    feats = w.features.view(np.int16) if spec.feat_dtype == "bf16" else w.features
    X = torch.as_tensor(feats).to(dev)
    labels = torch.as_tensor(w.labels).to(dev)
    seeds = [torch.as_tensor(s).to(dev) for s in w.seeds]
    torch.cuda.synchronize()
    upload_s = time.time() - t
    xdt = gnnhip.BF16 if spec.feat_dtype == "bf16" else gnnhip.F32
    shadow = (spec.shadow_fanout, spec.shadow_hops) if spec.shadow else None
    tr = gnnhip.Trainer(spec.kind, spec.dims, w.weights, spec.batch, spec.fanouts, w.graph.num_nodes,
                        xdt, dev, shadow=shadow)
    nb = len(seeds)

    def run(s, events=None):
        tr.step(csr, X, labels, seeds[s % nb], w.rng_key(s % nb), spec.lr, events=events)

    for s in range(args.warmup):
        run(s)
    torch.cuda.synchronize()
    assert gnnhip.check_errors() == 0
    _log(f"{spec.name}: warmup done ({args.warmup} steps)")

    # every launch of a few untimed steps, bracketed by events
    cap = 96
    cev = HipEvents(2 * cap * cal_steps)
    cal = []
    for c in range(cal_steps):
        tc = gnnhip.Trace(cev.ev[2 * cap * c: 2 * cap * (c + 1)])
        with tc:
            run(args.warmup + c)
        torch.cuda.synchronize()
        assert tc.dropped == 0, "trace capacity"
        names = tc.names()
        cal.append((names, [cev.elapsed_ms(2 * cap * c + 2 * i, 2 * cap * c + 2 * i + 1)
                            for i in range(len(names))]))
    cev.close()
    names = cal[0][0]
    assert all(n == names for n, _ in cal), "launch sequence changed between steps"
    keys = launch_keys(names)

    if args.pmc_child:
        # counters pass: the step sequence only, then the probes
        for s in range(args.steps):
            run(args.warmup + cal_steps + s)
        torch.cuda.synchronize()
        a = torch.ones(COPY_PROBE_FLOATS, device=dev)
        b = torch.empty_like(a)
        torch.mul(a, 1.0, out=b)
        del a, b
        for dt in (torch.float32, torch.bfloat16):
            g = torch.randn(GEMM_PROBE_N, GEMM_PROBE_N, device=dev).to(dt)
            torch.mm(g, g)
            del g
        torch.cuda.synchronize()
        assert gnnhip.check_errors() == 0
        with open(args.names_out, "w") as fh:
            json.dump(names, fh)
        _log(f"pmc child: {args.steps} steps of {len(names)} launches, probes done")
        return None

    cal_ms = {k: sum(d[i] for _, d in cal) / cal_steps for i, k in enumerate(keys)}
    modeled = {"gather", "aggregate", "gemm_fwd", "gemm_dw", "gemm_dx", "gemm_bwd", "scatter", "relu_mask",
               "softmax_xent", "sgd", "shadow_build", "shadow_emit", "head"}
    if not spec.shadow:
        modeled |= {"sample", "scans", "indices"}
    if spec.kind == "gat":
        modeled |= {"gat_scores", "gat_attend", "gat_attend_bwd", "gat_score_grad", "gat_colsum",
                    "gat_colsum_final"}
    dom = max((k for k in keys if k.split("#")[0] in modeled), key=lambda k: cal_ms[k])
    dom_name, dom_occ = dom.split("#")[0], int(dom.split("#")[1])
    occ_per_step = sum(1 for k in keys if k.split("#")[0] == dom_name)

    # the timed steps, with nothing recorded between launches
    first = args.warmup + cal_steps
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        run(first + i)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    elapsed_serial = t1 - t0
    assert gnnhip.check_errors() == 0
    _log(f"{spec.name}: timed {args.steps} serial steps in {elapsed_serial * 1e3:.1f} ms")

    # the same K steps pipelined: batch i + 1 is sampled on a second stream
    # while batch i trains (block slots alternate; every step still samples,
    # trains and updates the weights inside the timed region)
    batches = [(seeds[(first + i) % nb], w.rng_key((first + i) % nb)) for i in range(args.steps)]
    samp_stream = torch.cuda.Stream()
    tr.run_pipelined(csr, X, labels, batches[:2], spec.lr, sample_stream=samp_stream)  # untimed
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    tr.run_pipelined(csr, X, labels, batches, spec.lr, sample_stream=samp_stream)
    t_enq = time.perf_counter()
    torch.cuda.synchronize()
    elapsed_pipe = time.perf_counter() - t0
    enqueue_pipe = t_enq - t0
    assert gnnhip.check_errors() == 0
    _log(f"{spec.name}: timed {args.steps} pipelined steps in {elapsed_pipe * 1e3:.1f} ms")
    elapsed = elapsed_serial if args.serial else elapsed_pipe

    # the same steps again with stage events and events around the dominant
    # kernel's launches (recording events adds gaps, so these steps do not
    # enter the throughput)
    ns = len(gnnhip.STAGES)
    ev = HipEvents(2 * ns * args.steps)
    per_step = (ctypes.c_void_p * (2 * ns))
    ev_sets = [per_step(*ev.ev[2 * ns * i: 2 * ns * (i + 1)]) for i in range(args.steps)]
    tev = HipEvents(2 * occ_per_step * args.steps)
    dtrace = gnnhip.Trace(tev.ev, only=dom_name)
    with dtrace:
        for i in range(args.steps):
            run(first + i, ev_sets[i])
    torch.cuda.synchronize()
    assert gnnhip.check_errors() == 0
    assert dtrace.count == occ_per_step * args.steps and dtrace.dropped == 0
    stage_ms = {}
    for k, name in enumerate(gnnhip.STAGES):
        tot = sum(ev.elapsed_ms(2 * ns * i + 2 * k, 2 * ns * i + 2 * k + 1) for i in range(args.steps))
        stage_ms[name] = tot / args.steps
    ev.close()
    j = [i * occ_per_step + dom_occ for i in range(args.steps)]
    dom_ms = sum(tev.elapsed_ms(2 * x, 2 * x + 1) for x in j) / args.steps
    tev.close()

    # sizes of every timed step (sampling is deterministic: re-sample untimed)
    step_ids = [(first + i) % nb for i in range(args.steps)]
    edges = []
    if spec.shadow:
        deg = np.diff(w.graph.rowptr)
        un, ue, re_, rows = [], [], [], []
        for k, s in enumerate(step_ids):
            sub, cptr, ro = gnnhip.sample_shadow(csr, seeds[s], spec.shadow_fanout,
                                                 spec.shadow_hops, w.rng_key(s))
            c = sub.counts.cpu().numpy()
            r = ro.counts.cpu().numpy()
            edges.append(int(c[2]))
            un.append(int(c[1]))
            ue.append(int(c[2]))
            re_.append(int(r[2]))
            if k < 8:  # row words the extraction must read, from a few steps
                nodes = sub.src_nodes[: int(c[1])].cpu().numpy()
                rows.append(shadow_row_words(deg, nodes, cptr.cpu().numpy(), spec.batch))
        sz = {"union": (float(np.mean(un)), float(np.mean(ue))), "root_e": float(np.mean(re_)),
              "row_elems": float(np.mean(rows))}
    else:
        blocks = gnnhip.alloc_blocks(spec.batch, spec.fanouts, w.graph.num_nodes, dev)
        sws = torch.zeros(gnnhip.sample_workspace_bytes(spec.batch, spec.fanouts, w.graph.num_nodes),
                          dtype=torch.uint8, device=dev)
        hops = []
        for s in step_ids:
            gnnhip.sample_blocks(csr, seeds[s], spec.fanouts, w.rng_key(s), blocks, sws)
            c = torch.stack([b.counts for b in blocks]).cpu().numpy()
            edges.append(int(c[:, 2].sum()))
            hops.append(c[:, :3].astype(np.float64))
        sz = {"hops": [tuple(float(v) for v in x) for x in np.mean(hops, axis=0)]}
        del blocks, sws
    mean_edges = float(np.mean(edges))
    models = launch_models(spec, keys, sz)

    def peak_of(k):
        return MFMA_PEAK_TFLOPS[mfma_dtype(spec, k)] if models[k][0] == "mfma" else HBM_PEAK_GBS

    def rate(k, ms):
        b, a, _ = models[k]
        return a / (ms * 1e-3) / (1e9 if b == "hbm" else 1e12)

    def counters_of(k, ms):
        """Counter-based figures of launch k at duration ms, from the committed
        counters of the current kernel source (None if none)."""
        e = lookup_counters(cfg, k)
        if not e:
            return {}
        out = {"traffic": e["bytes"], "counter_frac": e["bytes"] / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS}
        fpm = mfma_flops_per_mop(cfg)
        if models[k][0] == "mfma" and fpm and "sq_insts_valu_mfma_mops_f32" in e:
            dt = mfma_dtype(spec, k)
            mops = e["sq_insts_valu_mfma_mops_bf16" if dt == "bf16" else "sq_insts_valu_mfma_mops_f32"]
            flops = mops * fpm[dt]
            out["mfma_flops"] = flops
            out["mfma_util"] = flops / (ms * 1e-3) / 1e12 / MFMA_PEAK_TFLOPS[dt]
        return out

    bound, amount, what = models[dom]
    achieved = rate(dom, dom_ms)
    peak = peak_of(dom)
    roofline = {"kernel": dom, "bound": bound, "achieved": achieved, "peak": peak,
                "unit": "GB/s" if bound == "hbm" else "TFLOP/s", "frac": achieved / peak,
                "traffic": None, "launch_ms": dom_ms, "algorithmic_per_launch": amount,
                "algorithmic": what}
    if bound == "mfma":
        roofline["mfma_dtype"] = mfma_dtype(spec, dom)
    roofline.update(counters_of(dom, dom_ms))
    roofline_all = {}
    for k in keys:
        if k not in models:
            continue
        r = {"bound": models[k][0], "ms": round(cal_ms[k], 5),
             "frac": round(rate(k, cal_ms[k]) / peak_of(k), 4)}
        c = counters_of(k, cal_ms[k])
        if "counter_frac" in c:
            r["counter_frac"] = round(c["counter_frac"], 4)
        if "mfma_util" in c:
            r["mfma_util"] = round(c["mfma_util"], 4)
        roofline_all[k] = r
    ga = [k for k in keys if k.split("#")[0] in ("gather", "aggregate")]
    ga_bytes = sum(models[k][1] for k in ga if k in models)
    ga_ms = sum(cal_ms[k] for k in ga)

    result = {
        "metric": "train mini-batches/sec",
        "value": args.steps / elapsed,
        "unit": "mini-batches/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": elapsed * 1e3 / args.steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": step_dtype(spec),
        "data": "synthetic",
        "config": {"workload": f"{spec.name}: {spec.graph} {w.graph.num_nodes} nodes "
                               f"{w.graph.num_edges} directed edges, {spec.kind} "
                               f"{'-'.join(map(str, spec.dims))}, "
                               + (f"ShaDow {spec.shadow_hops} hops x {spec.shadow_fanout}"
                                  if spec.shadow else f"fanouts {list(spec.fanouts)}")
                               + f", batch {spec.batch}, {spec.feat_dtype} features",
                   "global_batch": spec.batch,
                   "sampler": "shadow" if spec.shadow else "neighbor",
                   "parallelism": "single-gpu"},
        "sampled_edges_per_s": mean_edges * args.steps / elapsed,
        "schedule": "serial" if args.serial else "pipelined: sampling of batch i + 1 on a second "
                    "stream while batch i trains",
        "value_serial": args.steps / elapsed_serial,
        "value_pipelined": args.steps / elapsed_pipe,
        "host_enqueue_ms_per_step": enqueue_pipe * 1e3 / args.steps,
        "stage_ms": {k: round(v, 5) for k, v in stage_ms.items()},
        "roofline": roofline,
        "gather_aggregate": {"launches": ga, "algorithmic_bytes": ga_bytes, "ms": ga_ms,
                             "GB_per_s": ga_bytes / (ga_ms * 1e-3) / 1e9 if ga_ms else None,
                             "frac": ga_bytes / (ga_ms * 1e-3) / 1e9 / HBM_PEAK_GBS if ga_ms else None},
        "launch_ms": {k: round(cal_ms[k], 5) for k in keys},
        "roofline_all": roofline_all,
        "inputs": {"generation_s": round(gen_s, 1), "upload_s": round(upload_s, 1)},
    }
    if full:
        result["dlb"] = dlb_leg(gnnhip, torch, spec, csr, batches)
        _log(f"workload estimate: {result['dlb']['estimate_batches_per_s']:.0f} batches/s")
        if not spec.shadow and args.feature_cache == "on":
            fc = feature_cache_leg(gnnhip, torch, spec, w, csr, labels, seeds, args.steps, first, nb,
                                   dev)
            result["feature_cache"] = fc
            _log(f"host features: {fc['cache']['mini_batches_per_s']:.0f} mini-batches/s with the "
                 f"cache (hit rate {fc['cache']['hit_rate']:.2f}), "
                 f"{fc['zero_copy']['mini_batches_per_s']:.0f} reading every row in place")
    del tr, csr, X, labels, seeds
    torch.cuda.empty_cache()
    if full and not args.no_cpu_baseline:
        _log(f"cpu oracle baseline ({args.cpu_seconds:.0f} s budget)")
        done, cedges, cel = cpu_baseline(w, args.cpu_seconds)
        result["cpu_baseline"] = {
            "value": done / cel, "unit": "mini-batches/s", "cores": 1, "kind": "oracle",
            "sample": f"{done} consecutive training steps of the same workload (float64 oracle, "
                      f"single thread, {cel:.1f} s), {cedges / cel:.0f} sampled edges/s",
            "host": platform.processor() or platform.machine(), "host_cpus": os.cpu_count()}
    return result


def compact(r):
    """The figures of an extra workload kept in the headline's line."""
    keep = ("value", "value_serial", "value_pipelined", "ms_per_step", "sampled_edges_per_s",
            "dtype", "roofline", "gather_aggregate", "stage_ms")
    out = {k: r[k] for k in keep}
    out["workload"] = r["config"]["workload"]
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", type=int, default=5)
    ap.add_argument("--extra", default="2",
                    help="comma-separated workloads measured after the headline one (compact "
                         "figures under other_workloads; '' for none)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--feature-cache", choices=("on", "off"), default="on",
                    help="the host-resident-features leg (feature cache against zero-copy reads)")
    ap.add_argument("--serial", action="store_true",
                    help="report the serial loop (sampling and model pass of a step on one stream)")
    ap.add_argument("--traffic", action="store_true", help="measure counters with rocprofv3")
    ap.add_argument("--traffic-out", default=os.path.join(ROOT, "gpurun_out", "traffic.json"))
    ap.add_argument("--no-mfma-pass", action="store_true", help="--traffic: bytes only")
    ap.add_argument("--pmc-child", action="store_true", help=argparse.SUPPRESS)
    ap.add_argument("--names-out", default=None, help=argparse.SUPPRESS)
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); "
              "this benchmark has no multi-GPU path", file=sys.stderr)
        sys.exit(2)
    if args.traffic:
        measure_traffic(args)
        return
    result = measure(args.config, args, full=True)
    if args.pmc_child:
        return
    extras = [int(x) for x in args.extra.split(",") if x.strip()] if args.extra else []
    others = {}
    for cfg in extras:
        if cfg == args.config:
            continue
        from workloads import configs
        others[configs.CONFIGS[cfg].name] = compact(measure(cfg, args, full=False))
    if others:
        result["other_workloads"] = others
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
