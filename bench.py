"""Throughput of one neighbour-sampled GNN training step on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config 2]

Workload (default): 2-layer GraphSAGE-mean 100-256-47 on an R-MAT graph
(a, b, c, d = 0.57, 0.19, 0.19, 0.05) of 2,449,029 nodes and ~124M directed
edges (the shape of ogbn-products), fp32 N(0,1) features of width 100,
fanouts [25, 10], 1024 seeds per batch, SGD lr 0.01; batch s uses sampling
key 1 + s.  A step is the whole path: sampling + relabelling of both hops,
feature gather, forward, loss, backward, SGD, all inside the timed region with
every input resident in HBM.

Prints one JSON line: mini-batches/s, sampled edges/s, per-stage times, the
roofline of the dominant kernel, and the CPU oracle baseline.
"""
from __future__ import annotations

import argparse
import ctypes
import json
import os
import platform
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0      # MI355X HBM3E, AMD datasheet
FP32_MFMA_TFLOPS = 157.3   # MI355X dense fp32 matrix


def _log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


class HipEvents:
    """hipEvent_t handles from the HIP runtime already loaded by torch."""

    def __init__(self, n):
        self.rt = ctypes.CDLL("libamdhip64.so.7")
        self.rt.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.rt.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                                ctypes.c_void_p]
        self.rt.hipEventDestroy.argtypes = [ctypes.c_void_p]
        self.ev = (ctypes.c_void_p * n)()
        for i in range(n):
            h = ctypes.c_void_p()
            rc = self.rt.hipEventCreate(ctypes.byref(h))
            assert rc == 0, rc
            self.ev[i] = h.value

    def elapsed_ms(self, a, b):
        ms = ctypes.c_float()
        rc = self.rt.hipEventElapsedTime(ctypes.byref(ms), self.ev[a], self.ev[b])
        assert rc == 0, rc
        return ms.value

    def close(self):
        for i in range(len(self.ev)):
            self.rt.hipEventDestroy(self.ev[i])


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


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", type=int, default=2)
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); "
              "the multi-GPU path is not part of this build", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2403_17092_amd import gnnhip
    from workloads import configs

    spec = configs.CONFIGS[args.config]
    t = time.time()
    nsteps = args.warmup + args.steps
    w = configs.make_workload(spec, steps=min(spec.steps, nsteps) if spec.steps > 1 else 1)
    _log(f"workload {spec.name}: {w.graph.num_nodes} nodes, {w.graph.num_edges} edges "
         f"({time.time() - t:.1f} s)")
    dev = torch.device("cuda:0")
    rp = w.graph.rowptr if spec.rowptr64 else w.graph.rowptr.astype(np.int32)
    csr = gnnhip.Csr(torch.as_tensor(rp).to(dev), torch.as_tensor(w.graph.col).to(dev))
    feats = w.features.view(np.int16) if spec.feat_dtype == "bf16" else w.features
    X = torch.as_tensor(feats).to(dev)
    labels = torch.as_tensor(w.labels).to(dev)
    seeds = [torch.as_tensor(s).to(dev) for s in w.seeds]
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
    _log(f"warmup done ({args.warmup} steps)")

    ns = len(gnnhip.STAGES)
    ev = HipEvents(2 * ns * args.steps)
    per_step = (ctypes.c_void_p * (2 * ns))
    ev_sets = [per_step(*ev.ev[2 * ns * i: 2 * ns * (i + 1)]) for i in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        run(args.warmup + i, ev_sets[i])
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    elapsed = t1 - t0
    assert gnnhip.check_errors() == 0
    _log(f"timed {args.steps} steps in {elapsed * 1e3:.1f} ms")
    stage_ms = {}
    for k, name in enumerate(gnnhip.STAGES):
        tot = sum(ev.elapsed_ms(2 * ns * i + 2 * k, 2 * ns * i + 2 * k + 1) for i in range(args.steps))
        stage_ms[name] = tot / args.steps
    ev.close()

    # sizes of every timed step (sampling is deterministic: re-sample untimed)
    edges, n_outer, agg1_edges, n_dst1 = [], [], [], []
    if spec.shadow:
        for i in range(args.steps):
            s = (args.warmup + i) % nb
            sub, _, _ = gnnhip.sample_shadow(csr, seeds[s], spec.shadow_fanout, spec.shadow_hops,
                                             w.rng_key(s))
            c = sub.counts.cpu().numpy()
            edges.append(int(c[2]))
            n_outer.append(int(c[1]))
            agg1_edges.append(int(c[2]))
            n_dst1.append(int(c[0]))
    else:
        blocks = gnnhip.alloc_blocks(spec.batch, spec.fanouts, w.graph.num_nodes, dev)
        sws = torch.zeros(gnnhip.sample_workspace_bytes(spec.batch, spec.fanouts, w.graph.num_nodes),
                          dtype=torch.uint8, device=dev)
        for i in range(args.steps):
            s = (args.warmup + i) % nb
            gnnhip.sample_blocks(csr, seeds[s], spec.fanouts, w.rng_key(s), blocks, sws)
            c = torch.stack([b.counts for b in blocks]).cpu().numpy()
            edges.append(int(c[:, 2].sum()))
            n_outer.append(int(c[-1, 1]))
            agg1_edges.append(int(c[-1, 2]))
            n_dst1.append(int(c[-1, 0]))
    mean_edges = float(np.mean(edges))
    F = spec.feat_dim
    esz = 2 if spec.feat_dtype == "bf16" else 4
    # gather: read + write of every outer-frontier row, plus the ids
    gather_bytes = float(np.mean([n * (2 * F * esz + 4) for n in n_outer]))
    # layer-1 aggregation: every edge and every dst's own row read one input row
    # (the self row is copied next to the aggregate for SAGE, and is the self
    # edge for GCN); the GEMM input row written per dst (2F fp32 for SAGE, F for
    # GCN); indices and row pointers (and the per-edge degree for GCN)
    xw = 2 * F if spec.kind == "sage_mean" else F
    occ_b = 4 if spec.kind == "gcn" else 0
    agg_bytes = float(np.mean([(e + d) * F * esz + d * xw * 4 + 4 * (e + d + 1) + occ_b * (e + d)
                               for e, d in zip(agg1_edges, n_dst1)]))
    K1 = (2 if spec.kind == "sage_mean" else 1) * F
    gemm1_flops = float(np.mean([2.0 * d * K1 * spec.dims[1] for d in n_dst1]))
    cands = {
        "gather": ("hbm", gather_bytes / (stage_ms["gather"] * 1e-3) / 1e9, HBM_PEAK_GBS, "GB/s",
                   gather_bytes),
        "agg1": ("hbm", agg_bytes / (stage_ms["agg1"] * 1e-3) / 1e9, HBM_PEAK_GBS, "GB/s", agg_bytes),
        "gemm1": ("mfma", gemm1_flops / (stage_ms["gemm1"] * 1e-3) / 1e12, FP32_MFMA_TFLOPS,
                  "TFLOP/s", gemm1_flops),
    }
    dominant = max(cands, key=lambda k: stage_ms[k])
    bound, achieved, peak, unit, per_launch = cands[dominant]

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
        "dtype": "f32" if spec.feat_dtype == "f32" else "bf16-features/f32",
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
        "stage_ms": {k: round(v, 5) for k, v in stage_ms.items()},
        "roofline": {"kernel": dominant, "bound": bound, "achieved": achieved, "peak": peak,
                     "unit": unit, "frac": achieved / peak, "traffic": None,
                     "algorithmic_per_launch": per_launch},
        "roofline_all": {k: {"achieved": v[1], "unit": v[3], "frac": v[1] / v[2]}
                         for k, v in cands.items()},
    }
    if not args.no_cpu_baseline:
        _log(f"cpu oracle baseline ({args.cpu_seconds:.0f} s budget)")
        done, cedges, cel = cpu_baseline(w, args.cpu_seconds)
        result["cpu_baseline"] = {
            "value": done / cel, "unit": "mini-batches/s", "cores": 1, "kind": "oracle",
            "sample": f"{done} consecutive training steps of the same workload (float64 oracle, "
                      f"single thread, {cel:.1f} s), {cedges / cel:.0f} sampled edges/s",
            "host": platform.processor() or platform.machine(), "host_cpus": os.cpu_count()}
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
