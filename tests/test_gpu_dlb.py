"""GPU parity of the workload estimate (gnn_estimate_work,
gnn_shadow_estimate_work) against the oracle: bit-exact per-batch workloads
and edge counts, on small graphs, on the full-size configured workloads, and
against the blocks the training step itself samples."""
import numpy as np
import pytest
import torch

from oracle import dlb as odlb
from tests import gpu_common as gc
from tests import helpers
from workloads import configs, graphs

pytestmark = pytest.mark.gpu


def _estimate(csr, kind, dims, batches, B, fanouts=None, shadow=None):
    from paper_2403_17092_amd import gnnhip
    dev_batches = [(gc.seeds_to_device(s), k) for s, k in batches]
    work, edges = gnnhip.estimate_work(csr, kind, dims, dev_batches, B, fanouts=fanouts,
                                       shadow=shadow)
    torch.cuda.synchronize()
    assert gnnhip.check_errors() == 0
    return work.cpu().numpy(), edges.cpu().numpy()


@pytest.mark.parametrize("kind", ["sage_mean", "gcn", "gin", "gat"])
@pytest.mark.parametrize("fanouts", [(3,), (4, 2), (10, 5, 3), (64, 64)])
def test_estimate_small_graphs(kind, fanouts):
    rowptr, col = helpers.mixed_graph()
    dims = (8, 12, 8, 4)[: len(fanouts) + 1]
    batches = [(np.array([0, 46, 51, 43]), 5), (np.array([41, 3, 7]), 6), (np.array([51]), 7)]
    gc.announce("estimate", kind, fanouts, "mixed graph")
    csr = gc.csr_to_device(rowptr, col)
    for B in {len(b[0]) for b in batches}:
        sel = [b for b in batches if len(b[0]) == B]
        work, edges = _estimate(csr, kind, dims, sel, B, fanouts=fanouts)
        ow, oe = odlb.estimate_work(rowptr, col, [s for s, _ in sel], fanouts, [k for _, k in sel],
                                    kind, dims)
        np.testing.assert_array_equal(work, ow)
        np.testing.assert_array_equal(edges, oe)


@pytest.mark.parametrize("rowptr64", [False, True])
def test_estimate_power_law_many_batches(rowptr64):
    g = graphs.chunglu_graph(50_000, 20.0, 2.1, seed=3)
    B, fan, dims = 256, (15, 10, 5), (16, 32, 32, 8)
    batches = [(configs.make_seeds(g.num_nodes, B, 9, s), 100 + s) for s in range(12)]
    gc.announce("estimate power law, 12 batches, rowptr64", rowptr64)
    csr = gc.csr_to_device(g.rowptr, g.col, rowptr64)
    work, edges = _estimate(csr, "gcn", dims, batches, B, fanouts=fan)
    ow, oe = odlb.estimate_work(g.rowptr, g.col, [s for s, _ in batches], fan,
                                [k for _, k in batches], "gcn", dims)
    np.testing.assert_array_equal(work, ow)
    np.testing.assert_array_equal(edges, oe)
    assert len(set(work.tolist())) > 1  # the batches differ


@pytest.mark.parametrize("kind", ["sage_mean", "gcn", "gin", "gat"])
def test_shadow_estimate(kind):
    rowptr, col = helpers.random_graph(90, 0.12, 2)
    dims = (8, 12, 8, 4)
    g = np.random.Generator(np.random.PCG64(1))
    batches = [(g.permutation(90)[:20], 30 + s) for s in range(4)]
    gc.announce("shadow estimate", kind)
    csr = gc.csr_to_device(rowptr, col)
    work, edges = _estimate(csr, kind, dims, batches, 20, shadow=(4, 2))
    ow, oe = odlb.shadow_estimate_work(rowptr, col, [s for s, _ in batches], 4, 2,
                                       [k for _, k in batches], kind, dims)
    np.testing.assert_array_equal(work, ow)
    np.testing.assert_array_equal(edges, oe)


def test_estimate_no_batches():
    from paper_2403_17092_amd import gnnhip
    rowptr, col = helpers.path_graph(8)
    gc.announce("estimate, no batches")
    csr = gc.csr_to_device(rowptr, col)
    work, edges = gnnhip.estimate_work(csr, "sage_mean", (4, 4, 2), [], 4, fanouts=(2, 2))
    torch.cuda.synchronize()
    assert work.numel() == 0 and gnnhip.check_errors() == 0


def test_estimate_matches_the_training_steps_blocks():
    # the estimate samples exactly the blocks the training step trains on
    from paper_2403_17092_amd import gnnhip
    spec = configs.small_spec(num_nodes=6000, avg_degree=12.0, dims=(32, 24, 24, 7),
                              fanouts=(8, 5, 3), batch=64, steps=3)
    w = configs.make_workload(spec)
    dev = gc.device()
    csr = gc.csr_to_device(w.graph.rowptr, w.graph.col)
    X = torch.as_tensor(w.features).to(dev)
    labels = torch.as_tensor(w.labels).to(dev)
    tr = gnnhip.Trainer(spec.kind, spec.dims, w.weights, spec.batch, spec.fanouts,
                        w.graph.num_nodes, gnnhip.F32, dev)
    gc.announce("estimate vs training step blocks")
    work, edges = _estimate(csr, spec.kind, spec.dims,
                            [(w.seeds[s], w.rng_key(s)) for s in range(3)], spec.batch,
                            fanouts=spec.fanouts)
    L = spec.num_layers
    for s in range(3):
        tr.step(csr, X, labels, gc.seeds_to_device(w.seeds[s]), w.rng_key(s), spec.lr)
        got = tr.inspect()
        counts = [got["blocks"][h][:3] for h in range(L)]  # (n_dst, n_src, E) per hop
        assert edges[s].tolist() == [c[2] for c in counts]
        want = sum(counts[L - l][2] * spec.dims[l - 1] for l in range(1, L + 1))
        assert work[s] == want
    assert gnnhip.check_errors() == 0


@pytest.mark.parametrize("cfg", [2, 3, 4, 6, 7])
def test_estimate_full_configs(cfg):
    # the benchmark's workloads at full size, a few batches each
    spec = configs.CONFIGS[cfg]
    n = 2 if spec.shadow else 3  # the ShaDow oracle takes ~10 s per batch
    print(f"[dlb] config {cfg}: generating the graph", flush=True)
    g = configs.make_graph(spec)
    batches = [(configs.make_seeds(g.num_nodes, spec.batch, spec.seed_seed, s), 1 + s)
               for s in range(n)]
    gc.announce("estimate full config", cfg)
    csr = gc.csr_to_device(g.rowptr if spec.rowptr64 else g.rowptr.astype(np.int32), g.col)
    ids = [s for s, _ in batches]
    keys = [k for _, k in batches]
    if spec.shadow:
        work, edges = _estimate(csr, spec.kind, spec.dims, batches, spec.batch,
                                shadow=(spec.shadow_fanout, spec.shadow_hops))
        ow, oe = odlb.shadow_estimate_work(g.rowptr, g.col, ids, spec.shadow_fanout,
                                           spec.shadow_hops, keys, spec.kind, spec.dims)
    else:
        work, edges = _estimate(csr, spec.kind, spec.dims, batches, spec.batch,
                                fanouts=spec.fanouts)
        ow, oe = odlb.estimate_work(g.rowptr, g.col, ids, spec.fanouts, keys, spec.kind, spec.dims)
    np.testing.assert_array_equal(work, ow)
    np.testing.assert_array_equal(edges, oe)


def test_estimate_long_chain_of_sampling_calls():
    # consecutive sampling calls skip the sampler's begin launch except every
    # 1024th; 1030 batches cross that boundary, each still matching the oracle
    g = graphs.chunglu_graph(3000, 8.0, 2.1, seed=5)
    B, fan, dims = 32, (6, 4), (8, 8, 4)
    n = 1030
    batches = [(configs.make_seeds(g.num_nodes, B, 21, s), 500 + s) for s in range(n)]
    gc.announce("estimate, chain of", n, "sampling calls")
    csr = gc.csr_to_device(g.rowptr, g.col)
    work, edges = _estimate(csr, "sage_mean", dims, batches, B, fanouts=fan)
    ow, oe = odlb.estimate_work(g.rowptr, g.col, [s for s, _ in batches], fan,
                                [k for _, k in batches], "sage_mean", dims)
    np.testing.assert_array_equal(work, ow)
    np.testing.assert_array_equal(edges, oe)
