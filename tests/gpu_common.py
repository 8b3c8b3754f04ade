"""Helpers shared by the GPU parity tests (imported only by tests marked gpu)."""
from __future__ import annotations

import sys

import numpy as np
import torch

from oracle import model as omodel
from paper_2403_17092_amd import gnnhip

# Tolerances (normwise relative error; see helpers.assert_close)
TOL_FWD = 1e-4    # fp32 forward: agg, activations, logits, loss
TOL_GRAD = 1e-3   # fp32 gradients
TOL_BF16 = 2e-2   # runs with bfloat16 features
TOL_W = 1e-4      # fp32 weights after an SGD step


def announce(*what):
    """Name the case on stdout before any GPU work (flushed)."""
    print("[gpu case]", *what, flush=True)
    sys.stdout.flush()


def device():
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    return torch.device("cuda:0")


def csr_to_device(rowptr, col, rowptr64=False, scan_order=0, hub_degree=0) -> gnnhip.Csr:
    dev = device()
    rp = torch.as_tensor(np.asarray(rowptr, dtype=np.int64 if rowptr64 else np.int32)).to(dev)
    cl = torch.as_tensor(np.asarray(col, dtype=np.int32)).to(dev)
    return gnnhip.Csr(rp, cl, scan_order, hub_degree)


def seeds_to_device(seeds) -> torch.Tensor:
    return torch.as_tensor(np.asarray(seeds, dtype=np.int32)).to(device())


def compare_block(gpu_host, ob, what=""):
    """Bit-exact comparison of a GPU block (Block.host() tuple) with an oracle block."""
    nd, ns, ne, indptr, indices, src_nodes, src_occ = gpu_host
    assert (nd, ns, ne) == (ob.n_dst, ob.n_src, ob.n_edges), (what, (nd, ns, ne),
                                                               (ob.n_dst, ob.n_src, ob.n_edges))
    np.testing.assert_array_equal(indptr, ob.indptr, err_msg=f"{what} indptr")
    np.testing.assert_array_equal(indices, ob.indices, err_msg=f"{what} indices")
    np.testing.assert_array_equal(src_nodes, ob.src_nodes, err_msg=f"{what} src_nodes")
    np.testing.assert_array_equal(src_occ, omodel.out_degree(ob), err_msg=f"{what} src_occ")
