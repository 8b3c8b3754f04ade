"""GPU parity of neighbour sampling and relabelling: bit-exact against the oracle."""
import numpy as np
import pytest
import torch

from oracle import sampling
from tests import gpu_common as gc
from tests import helpers
from workloads import configs, graphs

pytestmark = pytest.mark.gpu


def _run(rowptr, col, seeds, fanouts, key, rowptr64=False, scan_order=0):
    gc.announce("sample", len(seeds), "seeds", list(fanouts), "key", key, "n", len(rowptr) - 1,
                "rowptr64", rowptr64, "scan_order", scan_order)
    from paper_2403_17092_amd import gnnhip
    csr = gc.csr_to_device(rowptr, col, rowptr64, scan_order=scan_order)
    blocks = gnnhip.sample_blocks(csr, gc.seeds_to_device(seeds), fanouts, key)
    torch.cuda.synchronize()
    assert gnnhip.check_errors() == 0
    ref = sampling.sample_blocks(rowptr, col, seeds, fanouts, key)
    for h, (gb, ob) in enumerate(zip(blocks, ref)):
        gc.compare_block(gb.host(), ob, f"hop {h + 1}")
    return blocks


@pytest.mark.parametrize("fanouts", [[5, 3, 2], [1], [64, 1], [2, 2, 2, 2]])
@pytest.mark.parametrize("key", [1, 12345])
def test_hand_graph(fanouts, key):
    rowptr, col = helpers.mixed_graph()
    _run(rowptr, col, np.array([0, 46, 51, 43, 41, 7]), fanouts, key)


def test_hub_max_fanout():
    rowptr, col = helpers.star_graph(1000)
    _run(rowptr, col, np.array([0, 5, 999]), [64, 64], 3)


def test_random_small_graphs():
    for seed in range(4):
        rowptr, col = helpers.random_graph(80, 0.15, seed)
        seeds = np.random.Generator(np.random.PCG64(seed)).permutation(80)[:17]
        _run(rowptr, col, seeds, [4, 3, 2], seed + 1)


def test_tiny_workload_full():
    w = configs.make_workload(1, with_features=False)
    g = w.graph
    _run(g.rowptr, g.col, w.seeds[0], w.spec.fanouts, 1)


@pytest.mark.parametrize("rowptr64", [False, True])
def test_mid_chunglu_many_partitions(rowptr64):
    # 1024 seeds, three hops: the last hop spans many partitions and scan tiles
    g = graphs.chunglu_graph(200_000, 20.0, 2.1, seed=77)
    seeds = configs.make_seeds(g.num_nodes, 1024, 5, 0)
    _run(g.rowptr, g.col, seeds, [15, 10, 5], 9, rowptr64)


def test_mid_chunglu_ticket_ordered_scans():
    # the same hops with every scan tile taken by ticket (the order large
    # grids use); the blocks must not change
    g = graphs.chunglu_graph(200_000, 20.0, 2.1, seed=77)
    seeds = configs.make_seeds(g.num_nodes, 1024, 5, 0)
    _run(g.rowptr, g.col, seeds, [15, 10, 5], 9, False, scan_order=1)


def test_deterministic_across_runs():
    from paper_2403_17092_amd import gnnhip
    g = graphs.chunglu_graph(50_000, 15.0, 2.1, seed=3)
    seeds = gc.seeds_to_device(configs.make_seeds(g.num_nodes, 512, 1, 0))
    csr = gc.csr_to_device(g.rowptr, g.col)
    gc.announce("determinism")
    a = [b.host() for b in gnnhip.sample_blocks(csr, seeds, [10, 10], 4)]
    b = [b.host() for b in gnnhip.sample_blocks(csr, seeds, [10, 10], 4)]
    for x, y in zip(a, b):
        for u, v in zip(x, y):
            np.testing.assert_array_equal(u, v)


def test_empty_batch():
    from paper_2403_17092_amd import gnnhip
    rowptr, col = helpers.mixed_graph()
    csr = gc.csr_to_device(rowptr, col)
    gc.announce("empty batch")
    seeds = torch.zeros(0, dtype=torch.int32, device=gc.device())
    blocks = gnnhip.sample_blocks(csr, seeds, [3, 2], 1)
    for b in blocks:
        nd, ns, ne = b.host()[:3]
        assert (nd, ns, ne) == (0, 0, 0)


def test_out_of_range_seed_sets_device_error():
    from paper_2403_17092_amd import gnnhip
    rowptr, col = helpers.mixed_graph()
    csr = gc.csr_to_device(rowptr, col)
    gc.announce("seed out of range")
    seeds = gc.seeds_to_device([0, 52, 3])  # 52 == N
    blocks = gnnhip.sample_blocks(csr, seeds, [3], 1)
    bits = gnnhip.check_errors()
    assert bits & gnnhip.DEVERR_SEED_RANGE
    nd, ns, ne, indptr = blocks[0].host()[:4]
    assert indptr[2] - indptr[1] == 0  # the bad seed has no edges
    assert gnnhip.check_errors() == 0  # cleared


def test_workspace_reuse_across_calls():
    # one workspace and one set of blocks for calls on two graphs (the second
    # smaller), several keys and seed batches: the per-node state carried
    # between calls must never leak into a later result
    from paper_2403_17092_amd import gnnhip
    ga = graphs.chunglu_graph(30_000, 12.0, 2.1, seed=21)
    gb = graphs.chunglu_graph(9_000, 25.0, 2.1, seed=22)
    fanouts = [8, 4]
    blocks = gnnhip.alloc_blocks(256, fanouts, ga.num_nodes, gc.device())
    ws = torch.zeros(gnnhip.sample_workspace_bytes(256, fanouts, ga.num_nodes), dtype=torch.uint8,
                     device=gc.device())
    for i, (g, key, batch) in enumerate([(ga, 1, 0), (ga, 2, 1), (gb, 3, 0), (ga, 1, 0), (gb, 3, 2)]):
        gc.announce("workspace reuse", i, "n", g.num_nodes, "key", key)
        seeds = configs.make_seeds(g.num_nodes, 256, 8, batch)
        csr = gc.csr_to_device(g.rowptr, g.col)
        got = gnnhip.sample_blocks(csr, gc.seeds_to_device(seeds), fanouts, key, blocks, ws)
        torch.cuda.synchronize()
        assert gnnhip.check_errors() == 0
        ref = sampling.sample_blocks(g.rowptr, g.col, seeds, fanouts, key)
        for h, (x, y) in enumerate(zip(got, ref)):
            gc.compare_block(x.host(), y, f"call {i} hop {h + 1}")


def test_bad_neighbour_id_sets_graph_error():
    from paper_2403_17092_amd import gnnhip
    # node 1's only neighbour is 7, outside [0, 3)
    rowptr = np.array([0, 2, 3, 4], np.int64)
    col = np.array([1, 2, 7, 0], np.int32)
    csr = gc.csr_to_device(rowptr, col)
    gc.announce("bad neighbour id")
    blocks = gnnhip.sample_blocks(csr, gc.seeds_to_device([1, 0]), [2, 2], 5)
    bits = gnnhip.check_errors()
    assert bits & gnnhip.DEVERR_GRAPH
    assert gnnhip.check_errors() == 0  # cleared
