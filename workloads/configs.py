"""The synthetic training workloads and their seeded inputs.

Every input of a training step -- graph, features, labels, seed batches,
initial weights -- is produced here from fixed keys, so the CPU oracle and the
GPU library see the same numbers.  The per-step sampling key is 1 + step.

Workloads (sizes follow the paper's evaluation setup, section 5.1.2 and
Table 2, with synthetic power-law graphs standing in for its datasets):

1. tiny:   Chung-Lu (gamma 2.1) 10,000 nodes, avg degree 10; fp32 F=128;
           GraphSAGE-mean 128-128-16; fanouts [10, 5]; batch 256; 1 step.
2. sage2:  R-MAT (0.57, 0.19, 0.19, 0.05), 2,449,029 nodes, ~124M directed
           edges (ogbn-products' shape); fp32 F=100; GraphSAGE-mean 100-256-47;
           fanouts [25, 10]; batch 1024; 100 steps.
3. gcn3:   R-MAT, 5M nodes, avg degree 50; fp32 F=128; GCN 128-256-256-64;
           fanouts [15, 10, 5]; batch 1024; 100 steps.
4. shadow: Chung-Lu (gamma 2.1), 2,449,029 nodes, avg degree 50; fp32 F=100;
           2-hop fanout-10 ShaDow subgraphs; GraphSAGE-mean 100-256-256-47;
           batch 1024 roots; 100 steps.
5. big:    R-MAT, 111M nodes, avg degree 30 (int64 row pointers); bf16 F=128;
           GraphSAGE-mean 128-256-256-172; fanouts [15, 10, 5]; batch 1024; 50 steps.
6. gin2:   sage2's graph with GIN-0 100-256-47 (each layer's MLP two products,
           the second [dims[l] x dims[l]]); fp32 F=100; fanouts [25, 10];
           batch 1024; 100 steps.
7. gat2:   sage2's graph with a one-head GAT 100-256-47; fp32 F=100; fanouts
           [25, 10]; batch 1024; 100 steps.
"""
from __future__ import annotations

import dataclasses
import os
from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np

from . import graphs

SAGE_MEAN = "sage_mean"
GCN = "gcn"
GIN = "gin"
GAT = "gat"


@dataclass(frozen=True)
class ConfigSpec:
    name: str
    graph: str            # "rmat" | "chunglu"
    num_nodes: int
    avg_degree: float
    n_pairs: int          # generator pairs (R-MAT) -- calibrated to the target edge count
    oversample: float     # Chung-Lu pair oversampling (duplicates and self loops are dropped)
    feat_dim: int
    feat_dtype: str       # "f32" | "bf16"
    kind: str             # SAGE_MEAN | GCN | GIN | GAT
    dims: tuple           # (F, hidden..., C)
    fanouts: tuple        # hop order: fanouts[0] is the seeds' budget
    batch: int
    steps: int
    shadow: bool = False
    shadow_hops: int = 0
    shadow_fanout: int = 0
    rowptr64: bool = False
    graph_seed: int = 0
    feat_seed: int = 0
    label_seed: int = 0
    seed_seed: int = 0
    weight_seed: int = 0
    lr: float = 0.01

    @property
    def num_classes(self) -> int:
        return self.dims[-1]

    @property
    def num_layers(self) -> int:
        return len(self.dims) - 1


CONFIGS = {
    1: ConfigSpec("tiny", "chunglu", 10_000, 10.0, 0, 1.016, 128, "f32", SAGE_MEAN, (128, 128, 16),
                  (10, 5), 256, 1, graph_seed=101, feat_seed=102, label_seed=103, seed_seed=104,
                  weight_seed=105),
    2: ConfigSpec("sage2", "rmat", 2_449_029, 0.0, 83_600_000, 1.0, 100, "f32", SAGE_MEAN,
                  (100, 256, 47), (25, 10), 1024, 100, graph_seed=201, feat_seed=202, label_seed=203,
                  seed_seed=204, weight_seed=205),
    3: ConfigSpec("gcn3", "rmat", 5_000_000, 0.0, 172_000_000, 1.0, 128, "f32", GCN,
                  (128, 256, 256, 64), (15, 10, 5), 1024, 100, graph_seed=301, feat_seed=302,
                  label_seed=303, seed_seed=304, weight_seed=305),
    4: ConfigSpec("shadow", "chunglu", 2_449_029, 50.0, 0, 1.006, 100, "f32", SAGE_MEAN,
                  (100, 256, 256, 47), (), 1024, 100, shadow=True, shadow_hops=2, shadow_fanout=10,
                  graph_seed=401, feat_seed=402, label_seed=403, seed_seed=404, weight_seed=405),
    6: ConfigSpec("gin2", "rmat", 2_449_029, 0.0, 83_600_000, 1.0, 100, "f32", GIN,
                  (100, 256, 47), (25, 10), 1024, 100, graph_seed=201, feat_seed=602, label_seed=603,
                  seed_seed=604, weight_seed=605),
    7: ConfigSpec("gat2", "rmat", 2_449_029, 0.0, 83_600_000, 1.0, 100, "f32", GAT,
                  (100, 256, 47), (25, 10), 1024, 100, graph_seed=201, feat_seed=702, label_seed=703,
                  seed_seed=704, weight_seed=705),
    5: ConfigSpec("big", "rmat", 111_000_000, 0.0, 1_754_000_000, 1.0, 128, "bf16", SAGE_MEAN,
                  (128, 256, 256, 172), (15, 10, 5), 1024, 50, rowptr64=True, graph_seed=501,
                  feat_seed=502, label_seed=503, seed_seed=504, weight_seed=505),
}


def make_graph(spec: ConfigSpec, log=graphs._quiet) -> graphs.CSRGraph:
    if spec.graph == "rmat":
        return graphs.rmat_graph(spec.num_nodes, spec.n_pairs, spec.graph_seed, log=log)
    return graphs.chunglu_graph(spec.num_nodes, spec.avg_degree, 2.1, spec.graph_seed, spec.oversample,
                                log=log)


def make_labels(n: int, num_classes: int, seed: int) -> np.ndarray:
    return np.random.Generator(np.random.PCG64([seed, 1])).integers(
        0, num_classes, size=n, dtype=np.int32)


def make_seeds(n: int, batch: int, seed: int, step: int) -> np.ndarray:
    """Batch of `batch` distinct node ids, uniform without replacement."""
    g = np.random.Generator(np.random.PCG64([seed, 2, step]))
    return g.choice(n, size=batch, replace=False).astype(np.int32)


def weight_shapes(kind: str, dims) -> List[tuple]:
    """Flat parameter order: per layer l = 1..L, SAGE stores W_self then W_neigh,
    GCN stores W, each [dims[l-1] x dims[l]]; GIN stores W_a [dims[l-1] x
    dims[l]] then W_b [dims[l] x dims[l]]; GAT stores W [dims[l-1] x dims[l]]
    then the attention vectors a [2 x dims[l]].  All row-major."""
    shapes = []
    for l in range(1, len(dims)):
        if kind == SAGE_MEAN:
            shapes += [(dims[l - 1], dims[l]), (dims[l - 1], dims[l])]
        elif kind == GIN:
            shapes += [(dims[l - 1], dims[l]), (dims[l], dims[l])]
        elif kind == GAT:
            shapes += [(dims[l - 1], dims[l]), (2, dims[l])]
        else:
            shapes += [(dims[l - 1], dims[l])]
    return shapes


def make_weights(kind: str, dims, seed: int) -> List[np.ndarray]:
    """Glorot-uniform initial weights, float32."""
    g = np.random.Generator(np.random.PCG64([seed, 3]))
    out = []
    for (fi, fo) in weight_shapes(kind, dims):
        a = np.sqrt(6.0 / (fi + fo))
        out.append(g.uniform(-a, a, size=(fi, fo)).astype(np.float32))
    return out


@dataclass
class Workload:
    spec: ConfigSpec
    graph: graphs.CSRGraph
    features: np.ndarray          # [N x F] float32 or uint16 (bf16 bits)
    labels: np.ndarray            # int32 [N]
    weights: List[np.ndarray]     # float32, weight_shapes order
    seeds: List[np.ndarray] = field(default_factory=list)  # per step, int32 [B]

    def rng_key(self, step: int) -> int:
        return 1 + step


def make_workload(cfg: int | ConfigSpec, steps: Optional[int] = None, graph=None,
                  with_features: bool = True, log=graphs._quiet) -> Workload:
    """Graph, features, labels, initial weights and per-step seed batches; `log`
    receives one line per finished generation stage."""
    spec = CONFIGS[cfg] if isinstance(cfg, int) else cfg
    g = make_graph(spec, log) if graph is None else graph
    n = g.num_nodes
    feats = (graphs.normal_features(n, spec.feat_dim, spec.feat_seed, spec.feat_dtype)
             if with_features else None)
    if with_features:
        log(f"generated {n} x {spec.feat_dim} {spec.feat_dtype} features")
    labels = make_labels(n, spec.num_classes, spec.label_seed)
    weights = make_weights(spec.kind, spec.dims, spec.weight_seed)
    nsteps = spec.steps if steps is None else steps
    seeds = [make_seeds(n, spec.batch, spec.seed_seed, s) for s in range(nsteps)]
    return Workload(spec, g, feats, labels, weights, seeds)


def small_spec(**kw) -> ConfigSpec:
    """A small custom configuration for tests (defaults: Chung-Lu 2,000 nodes)."""
    base = dict(name="small", graph="chunglu", num_nodes=2000, avg_degree=8.0, n_pairs=0,
                oversample=1.0, feat_dim=32, feat_dtype="f32", kind=SAGE_MEAN, dims=(32, 16, 8),
                fanouts=(6, 4), batch=64, steps=1, graph_seed=11, feat_seed=12, label_seed=13,
                seed_seed=14, weight_seed=15)
    base.update(kw)
    if "feat_dim" not in kw:
        base["feat_dim"] = base["dims"][0]
    return ConfigSpec(**base)
