"""GPU parity of the gather, the layers and the whole training step against the
oracle (bit-exact integer outputs, tolerance-matched floating point)."""
import ctypes

import numpy as np
import pytest
import torch

from oracle import model as omodel
from oracle import sampling
from tests import gpu_common as gc
from tests import helpers
from workloads import configs, graphs

pytestmark = pytest.mark.gpu


def _feat_tensor(feats):
    dev = gc.device()
    if feats.dtype == np.uint16:
        return torch.as_tensor(feats.view(np.int16)).to(dev)
    return torch.as_tensor(feats).to(dev)


@pytest.mark.parametrize("dtype,F", [("f32", 100), ("f32", 4), ("bf16", 128), ("bf16", 8)])
def test_gather_bit_exact(dtype, F):
    from paper_2403_17092_amd import gnnhip
    gc.announce("gather", dtype, F)
    n = 5000
    X = graphs.normal_features(n, F, 3, dtype)
    ids = np.random.Generator(np.random.PCG64(1)).integers(0, n, 3001).astype(np.int32)
    Xd = _feat_tensor(X)
    idd = torch.as_tensor(ids).to(gc.device())
    cnt = torch.tensor([3001, 0, 0, 0], dtype=torch.int32, device=gc.device())
    out = gnnhip.gather_features(Xd, idd, cnt, 3100)
    torch.cuda.synchronize()
    got = out[:3001].cpu().numpy()
    if dtype == "bf16":
        got = got.view(np.uint16)
    np.testing.assert_array_equal(got, X[ids])
    assert gnnhip.check_errors() == 0


def _layer_setup(kind, F_in, F_out, seed, in_dtype="f32"):
    """A sampled block on a Chung-Lu graph plus random inputs and weights."""
    g = graphs.chunglu_graph(20_000, 12.0, 2.1, seed=seed)
    seeds = configs.make_seeds(g.num_nodes, 700, seed, 0)
    blocks = sampling.sample_blocks(g.rowptr, g.col, seeds, [12, 6], seed + 1)
    ob = blocks[1]  # the outer hop: the block layer 1 runs on
    rng = np.random.Generator(np.random.PCG64(seed))
    if in_dtype == "bf16":
        H = graphs.normal_features(ob.n_src, F_in, seed, "bf16")
    else:
        H = rng.normal(size=(ob.n_src, F_in)).astype(np.float32)
    Ws = rng.normal(0, 0.2, (F_in, F_out)).astype(np.float32)
    Wn = rng.normal(0, 0.2, (F_in, F_out)).astype(np.float32)
    dZ = rng.normal(size=(ob.n_dst, F_out)).astype(np.float32)
    return g, seeds, blocks, ob, H, Ws, Wn, dZ


def _stacked(kind, Ws, Wn):
    return np.concatenate([Ws, Wn], axis=0) if kind == "sage_mean" else Wn


def _x_ref(kind, A, H64, n_dst):
    agg = A @ H64
    return np.concatenate([H64[:n_dst], agg], axis=1) if kind == "sage_mean" else agg


@pytest.mark.parametrize("kind", ["sage_mean", "gcn"])
@pytest.mark.parametrize("F_in,F_out", [(100, 256), (256, 47), (128, 16), (4, 5)])
def test_layer_forward_backward(kind, F_in, F_out):
    from paper_2403_17092_amd import gnnhip
    gc.announce("layer", kind, F_in, F_out)
    g, seeds, blocks, ob, H, Ws, Wn, dZ = _layer_setup(kind, F_in, F_out, 5)
    csr = gc.csr_to_device(g.rowptr, g.col)
    gb = gnnhip.sample_blocks(csr, gc.seeds_to_device(seeds), [12, 6], 6)
    gc.compare_block(gb[1].host(), ob, "outer block")
    dev = gc.device()
    k = gnnhip.KIND[kind]
    W = _stacked(kind, Ws, Wn)
    Hd = torch.as_tensor(H).to(dev)
    Wd = torch.as_tensor(W).to(dev)
    X, Hout = gnnhip.layer_fwd(gb[1], k, Hd, Wd, relu=True)
    # oracle
    A = omodel.agg_matrix(ob, kind)
    H64 = H.astype(np.float64)
    rX = _x_ref(kind, A, H64, ob.n_dst)
    Z = rX @ W.astype(np.float64)
    torch.cuda.synchronize()
    helpers.assert_close(X[: ob.n_dst].cpu().numpy(), rX, gc.TOL_FWD, "X")
    helpers.assert_close(Hout[: ob.n_dst].cpu().numpy(), np.maximum(Z, 0), gc.TOL_FWD, "H_out")
    # backward with input gradient and ReLU mask of the input (H > 0)
    Hpos = np.maximum(H, 0).astype(np.float32)
    Hpd = torch.as_tensor(Hpos).to(dev)
    X2, _ = gnnhip.layer_fwd(gb[1], k, Hpd, Wd, relu=False)
    dZd = torch.as_tensor(dZ).to(dev)
    dW, dH = gnnhip.layer_bwd(gb[1], k, F_in, X2, Hpd, Wd, dZd, want_dH=True, mask_relu=True)
    torch.cuda.synchronize()
    Hp64 = Hpos.astype(np.float64)
    rX2 = _x_ref(kind, A, Hp64, ob.n_dst)
    dZ64 = dZ.astype(np.float64)
    helpers.assert_close(dW.cpu().numpy(), rX2.T @ dZ64, gc.TOL_GRAD, "dW")
    rdH = A.T @ (dZ64 @ Wn.T.astype(np.float64))
    if kind == "sage_mean":
        rdH[: ob.n_dst] += dZ64 @ Ws.T.astype(np.float64)
    rdH = rdH * (Hp64 > 0)
    helpers.assert_close(dH[: ob.n_src].cpu().numpy(), rdH, gc.TOL_GRAD, "dH_in")
    assert gnnhip.check_errors() == 0


@pytest.mark.parametrize("F_in,F_out", [(100, 256), (256, 47), (128, 16), (4, 5)])
def test_gin_layer_forward_backward(F_in, F_out):
    # X = [agg | M | pad] with M = relu(agg W_a); Z = M W_b; the backward goes
    # through both products and M's ReLU
    from paper_2403_17092_amd import gnnhip
    gc.announce("GIN layer", F_in, F_out)
    g, seeds, blocks, ob, H, Wa, _, dZ = _layer_setup("gin", F_in, F_out, 7)
    Wb = np.random.Generator(np.random.PCG64(F_in * 1000 + F_out)).normal(
        0, 0.2, (F_out, F_out)).astype(np.float32)
    csr = gc.csr_to_device(g.rowptr, g.col)
    gb = gnnhip.sample_blocks(csr, gc.seeds_to_device(seeds), [12, 6], 8)
    gc.compare_block(gb[1].host(), ob, "outer block")
    dev = gc.device()
    W = np.concatenate([Wa, Wb], axis=0)
    Wd = torch.as_tensor(W).to(dev)
    X, Hout = gnnhip.layer_fwd(gb[1], gnnhip.GIN, torch.as_tensor(H).to(dev), Wd, relu=True)
    A = omodel.agg_matrix(ob, "gin")
    Wa64, Wb64 = Wa.astype(np.float64), Wb.astype(np.float64)
    agg = A @ H.astype(np.float64)
    M = np.maximum(agg @ Wa64, 0)
    torch.cuda.synchronize()
    assert X.shape[1] == F_in + (F_out + 3) // 4 * 4
    Xh = X[: ob.n_dst].cpu().numpy()
    helpers.assert_close(Xh[:, :F_in], agg, gc.TOL_FWD, "agg")
    helpers.assert_close(Xh[:, F_in: F_in + F_out], M, gc.TOL_FWD, "M")
    helpers.assert_close(Hout[: ob.n_dst].cpu().numpy(), np.maximum(M @ Wb64, 0), gc.TOL_FWD, "H_out")
    # backward with input gradient and ReLU mask of the input (H > 0)
    Hpos = np.maximum(H, 0).astype(np.float32)
    Hpd = torch.as_tensor(Hpos).to(dev)
    X2, _ = gnnhip.layer_fwd(gb[1], gnnhip.GIN, Hpd, Wd, relu=False)
    dW, dH = gnnhip.layer_bwd(gb[1], gnnhip.GIN, F_in, X2, Hpd, Wd, torch.as_tensor(dZ).to(dev),
                              want_dH=True, mask_relu=True)
    torch.cuda.synchronize()
    Hp64 = Hpos.astype(np.float64)
    agg2 = A @ Hp64
    P2 = agg2 @ Wa64
    dZ64 = dZ.astype(np.float64)
    dP = (dZ64 @ Wb64.T) * (P2 > 0)
    dWh = dW.cpu().numpy()
    helpers.assert_close(dWh[F_in:], np.maximum(P2, 0).T @ dZ64, gc.TOL_GRAD, "dW_b")
    helpers.assert_close(dWh[:F_in], agg2.T @ dP, gc.TOL_GRAD, "dW_a")
    rdH = (A.T @ (dP @ Wa64.T)) * (Hp64 > 0)
    helpers.assert_close(dH[: ob.n_src].cpu().numpy(), rdH, gc.TOL_GRAD, "dH_in")
    assert gnnhip.check_errors() == 0


def test_layer_forward_bf16_input():
    from paper_2403_17092_amd import gnnhip
    gc.announce("layer bf16")
    g, seeds, blocks, ob, H, Ws, Wn, dZ = _layer_setup("sage_mean", 128, 64, 7, "bf16")
    csr = gc.csr_to_device(g.rowptr, g.col)
    gb = gnnhip.sample_blocks(csr, gc.seeds_to_device(seeds), [12, 6], 8)
    dev = gc.device()
    Hd = _feat_tensor(H)
    W = _stacked("sage_mean", Ws, Wn)
    Wd = torch.as_tensor(W).to(dev)
    X, Hout = gnnhip.layer_fwd(gb[1], gnnhip.SAGE_MEAN, Hd, Wd, relu=False)
    dW, _ = gnnhip.layer_bwd(gb[1], gnnhip.SAGE_MEAN, 128, X, None, Wd, torch.as_tensor(dZ).to(dev),
                             want_dH=False, mask_relu=False)
    torch.cuda.synchronize()
    H64 = omodel.widen(H)
    A = omodel.agg_matrix(ob, "sage_mean")
    rX = _x_ref("sage_mean", A, H64, ob.n_dst)
    helpers.assert_close(X[: ob.n_dst].cpu().numpy(), rX, gc.TOL_BF16, "X")
    helpers.assert_close(Hout[: ob.n_dst].cpu().numpy(), rX @ W, gc.TOL_BF16, "Z")
    helpers.assert_close(dW.cpu().numpy(), rX.T @ dZ, gc.TOL_BF16, "dW")


def test_softmax_xent():
    from paper_2403_17092_amd import gnnhip
    gc.announce("softmax")
    rng = np.random.Generator(np.random.PCG64(2))
    for B, C in [(1024, 47), (256, 16), (7, 172), (3, 1)]:
        z = (rng.normal(size=(B, C)) * 3).astype(np.float32)
        y = rng.integers(0, C, B).astype(np.int32)
        dev = gc.device()
        loss, dl = gnnhip.softmax_xent(torch.as_tensor(z).to(dev), torch.as_tensor(y).to(dev))
        rl, rd = omodel.softmax_xent(z.astype(np.float64), y)
        torch.cuda.synchronize()
        assert abs(loss.item() - rl) <= gc.TOL_FWD * max(1.0, abs(rl))
        helpers.assert_close(dl.cpu().numpy(), rd, gc.TOL_GRAD, "dlogits")


def _train_parity(w, steps, tol_fwd, tol_grad, tol_w, rowptr64=False):
    """Run `steps` GPU training steps and the oracle side by side, comparing every
    intermediate of every step."""
    from paper_2403_17092_amd import gnnhip
    spec = w.spec
    dev = gc.device()
    csr = gc.csr_to_device(w.graph.rowptr, w.graph.col, rowptr64)
    X = _feat_tensor(w.features)
    labels = torch.as_tensor(w.labels).to(dev)
    xdt = gnnhip.BF16 if spec.feat_dtype == "bf16" else gnnhip.F32
    tr = gnnhip.Trainer(spec.kind, spec.dims, w.weights, spec.batch, spec.fanouts, w.graph.num_nodes,
                        xdt, dev)
    W = [x.astype(np.float64) for x in w.weights]
    for s in range(steps):
        gc.announce("train step", spec.name, s)
        seeds = gc.seeds_to_device(w.seeds[s])
        loss = tr.step(csr, X, labels, seeds, w.rng_key(s), spec.lr)
        got = tr.inspect()
        assert gnnhip.check_errors() == 0
        ref = omodel.train_step(w.graph.rowptr, w.graph.col, w.features, w.labels, w.seeds[s],
                                spec.fanouts, w.rng_key(s), spec.kind, W, spec.lr)
        for h, ob in enumerate(ref["blocks"]):
            gc.compare_block(got["blocks"][h], ob, f"step {s} hop {h + 1}")
        # no gathered copy: layer 1 reads the feature rows in place (its X is checked below)
        assert got["xg"] is None
        L = spec.num_layers
        for l in range(L):
            want_x = ref["agg"][l]
            if spec.kind == "sage_mean":
                want_x = np.concatenate([ref["H"][l][: want_x.shape[0]], want_x], axis=1)
            if spec.kind == "gin":
                # [agg | M | pad], M = relu(agg W_a)
                F_in, F_out = spec.dims[l], spec.dims[l + 1]
                helpers.assert_close(got["x"][l][:, F_in: F_in + F_out], np.maximum(ref["P"][l], 0),
                                     tol_fwd, f"step {s} M{l + 1}")
                got_x = got["x"][l][:, :F_in]
            else:
                got_x = got["x"][l]
            if spec.kind == "gat":
                # GAT keeps layer 1's input rows only: the gathered features
                if l == 0:
                    helpers.assert_close(got_x, ref["xg"][: got_x.shape[0]], 0.0, f"step {s} input rows")
                else:
                    assert got_x is None
            else:
                helpers.assert_close(got_x, want_x, tol_fwd, f"step {s} X{l + 1}")
            want_h = ref["H"][l + 1]
            helpers.assert_close(got["h"][l], want_h, tol_fwd, f"step {s} H{l + 1}")
        assert abs(loss.item() - ref["loss"]) <= tol_fwd * abs(ref["loss"]), (loss.item(), ref["loss"])
        dW = np.concatenate([g.ravel() for g in ref["dW"]])
        off = 0
        for i, g in enumerate(ref["dW"]):
            helpers.assert_close(got["dweights"][off: off + g.size], g.ravel(), tol_grad,
                                 f"step {s} dW[{i}]")
            off += g.size
        W = ref["W_new"]
        Wgot = tr.weights.cpu().numpy()
        helpers.assert_close(Wgot, np.concatenate([x.ravel() for x in W]), tol_w, f"step {s} W")
    return tr


def test_train_step_tiny_workload():
    w = configs.make_workload(1)
    _train_parity(w, 1, gc.TOL_FWD, gc.TOL_GRAD, gc.TOL_W)


@pytest.mark.parametrize("rowptr64", [False, True])
def test_train_steps_small_sage(rowptr64):
    spec = configs.small_spec(num_nodes=3000, dims=(32, 24, 7), fanouts=(6, 4), batch=96, steps=3)
    w = configs.make_workload(spec)
    _train_parity(w, 3, gc.TOL_FWD, gc.TOL_GRAD, gc.TOL_W, rowptr64)


def test_train_steps_small_gcn_three_layers():
    spec = configs.small_spec(num_nodes=4000, kind="gcn", dims=(16, 32, 20, 5), fanouts=(5, 4, 3),
                              batch=128, steps=2)
    w = configs.make_workload(spec)
    _train_parity(w, 2, gc.TOL_FWD, gc.TOL_GRAD, gc.TOL_W)


def test_train_steps_small_bf16_three_layers():
    spec = configs.small_spec(num_nodes=5000, feat_dtype="bf16", dims=(64, 32, 32, 11),
                              fanouts=(7, 5, 3), batch=200, steps=2, rowptr64=True)
    w = configs.make_workload(spec)
    _train_parity(w, 2, gc.TOL_BF16, gc.TOL_BF16, gc.TOL_BF16, rowptr64=True)


def test_train_steps_bf16_ragged_widths():
    # bf16 layer 1 whose widths are no multiple of the product tiles: 2 x 40
    # inputs (the last 32-wide k step half empty), 36 outputs (a partial
    # column tile); two layers, so the fused output layer's weight-gradient
    # partials and layer 1's are summed by the same optimizer launch
    spec = configs.small_spec(num_nodes=4000, feat_dtype="bf16", dims=(40, 36, 12), fanouts=(6, 4),
                              batch=150, steps=2)
    w = configs.make_workload(spec)
    _train_parity(w, 2, gc.TOL_BF16, gc.TOL_BF16, gc.TOL_BF16)


def test_train_steps_gcn_bf16_three_layers():
    # GCN on bf16 features: layer 1's products read agg alone (48 wide)
    spec = configs.small_spec(num_nodes=5000, kind="gcn", feat_dtype="bf16", dims=(48, 40, 24, 6),
                              fanouts=(6, 5, 3), batch=160, steps=2)
    w = configs.make_workload(spec)
    _train_parity(w, 2, gc.TOL_BF16, gc.TOL_BF16, gc.TOL_BF16)


def test_train_steps_wide_output_layer():
    # more classes than the fused output layer takes: separate GEMMs and loss
    spec = configs.small_spec(num_nodes=3000, dims=(32, 24, 72), fanouts=(6, 4), batch=90, steps=2)
    w = configs.make_workload(spec)
    _train_parity(w, 2, gc.TOL_FWD, gc.TOL_GRAD, gc.TOL_W)


def test_train_steps_single_layer():
    spec = configs.small_spec(num_nodes=3000, dims=(32, 10), fanouts=(5,), batch=50, steps=2)
    w = configs.make_workload(spec)
    _train_parity(w, 2, gc.TOL_FWD, gc.TOL_GRAD, gc.TOL_W)


def test_train_steps_head_in_two_parts():
    # 2 x 100 inputs: the output layer's blocks split the width in two parts
    # of 128 rows (the second ragged) and exchange their partial logits; a
    # ragged last row tile and padding tiles
    spec = configs.small_spec(num_nodes=3000, dims=(32, 100, 9), fanouts=(5, 4), batch=70, steps=2)
    w = configs.make_workload(spec)
    _train_parity(w, 2, gc.TOL_FWD, gc.TOL_GRAD, gc.TOL_W)


def test_train_steps_full_head_widths():
    # the fused output layer at its limits: 2 x 256 inputs, 64 classes, a
    # ragged last row tile
    spec = configs.small_spec(num_nodes=4000, dims=(16, 256, 64), fanouts=(4, 3), batch=70, steps=2)
    w = configs.make_workload(spec)
    _train_parity(w, 2, gc.TOL_FWD, gc.TOL_GRAD, gc.TOL_W)


def test_train_steps_small_gin():
    # GIN-0: sum aggregation with the self row, a two-product MLP per layer,
    # and an output layer that runs unfused
    spec = configs.small_spec(num_nodes=3000, kind="gin", dims=(32, 24, 7), fanouts=(6, 4), batch=96,
                              steps=3)
    w = configs.make_workload(spec)
    _train_parity(w, 3, gc.TOL_FWD, gc.TOL_GRAD, gc.TOL_W)


def test_train_steps_gin_bf16_three_layers():
    spec = configs.small_spec(num_nodes=5000, kind="gin", feat_dtype="bf16", dims=(64, 32, 32, 11),
                              fanouts=(7, 5, 3), batch=200, steps=2)
    w = configs.make_workload(spec)
    _train_parity(w, 2, gc.TOL_BF16, gc.TOL_BF16, gc.TOL_BF16)


def test_train_steps_small_gat():
    # one-head GAT: T = H W over the src rows, attention over the sampled
    # edges and the self edge, backward through the softmax
    spec = configs.small_spec(num_nodes=3000, kind="gat", dims=(32, 24, 7), fanouts=(6, 4), batch=96,
                              steps=3)
    w = configs.make_workload(spec)
    _train_parity(w, 3, gc.TOL_FWD, gc.TOL_GRAD, gc.TOL_W)


def test_train_steps_gat_bf16_three_layers():
    spec = configs.small_spec(num_nodes=5000, kind="gat", feat_dtype="bf16", dims=(64, 32, 32, 11),
                              fanouts=(7, 5, 3), batch=200, steps=2)
    w = configs.make_workload(spec)
    _train_parity(w, 2, gc.TOL_BF16, gc.TOL_BF16, gc.TOL_BF16)


def test_train_steps_gat_single_layer_wide_rows():
    # 72 classes: 18 lanes of 4 columns rounded up to 32; rows of 61-degree
    # power-law hubs need two sweeps of 64 edges with the self edge
    spec = configs.small_spec(num_nodes=3000, kind="gat", dims=(32, 72), fanouts=(64,), batch=50,
                              steps=2)
    w = configs.make_workload(spec)
    _train_parity(w, 2, gc.TOL_FWD, gc.TOL_GRAD, gc.TOL_W)


def test_train_steps_gin_single_layer():
    spec = configs.small_spec(num_nodes=3000, kind="gin", dims=(32, 10), fanouts=(5,), batch=50, steps=2)
    w = configs.make_workload(spec)
    _train_parity(w, 2, gc.TOL_FWD, gc.TOL_GRAD, gc.TOL_W)


def _pipelined_parity(spec, steps, tol_fwd, tol_w):
    """Steps run with the next batch sampled on a second stream while the
    current one trains (block slots alternating): every step's loss and the
    weights after the last match the oracle run step by step."""
    from paper_2403_17092_amd import gnnhip
    w = configs.make_workload(spec)
    dev = gc.device()
    csr = gc.csr_to_device(w.graph.rowptr, w.graph.col)
    X = _feat_tensor(w.features)
    labels = torch.as_tensor(w.labels).to(dev)
    xdt = gnnhip.BF16 if spec.feat_dtype == "bf16" else gnnhip.F32
    tr = gnnhip.Trainer(spec.kind, spec.dims, w.weights, spec.batch, spec.fanouts, w.graph.num_nodes,
                        xdt, dev)
    gc.announce("pipelined train steps", spec.name, steps)
    batches = [(gc.seeds_to_device(w.seeds[s]), w.rng_key(s)) for s in range(steps)]
    losses = tr.run_pipelined(csr, X, labels, batches, spec.lr)
    torch.cuda.synchronize()
    losses = losses.cpu()
    assert gnnhip.check_errors() == 0
    W = [x.astype(np.float64) for x in w.weights]
    for s in range(steps):
        ref = omodel.train_step(w.graph.rowptr, w.graph.col, w.features, w.labels, w.seeds[s],
                                spec.fanouts, w.rng_key(s), spec.kind, W, spec.lr)
        assert abs(losses[s].item() - ref["loss"]) <= tol_fwd * abs(ref["loss"]), (s, losses[s].item(),
                                                                                   ref["loss"])
        W = ref["W_new"]
    helpers.assert_close(tr.weights.cpu().numpy(), np.concatenate([x.ravel() for x in W]), tol_w,
                         f"weights after {steps} pipelined steps")


def test_pipelined_steps_sage():
    spec = configs.small_spec(num_nodes=3000, dims=(32, 24, 7), fanouts=(6, 4), batch=96, steps=5)
    _pipelined_parity(spec, 5, gc.TOL_FWD, gc.TOL_W)


def test_pipelined_steps_gcn_three_layers():
    spec = configs.small_spec(num_nodes=4000, kind="gcn", dims=(16, 32, 20, 5), fanouts=(5, 4, 3),
                              batch=128, steps=4)
    _pipelined_parity(spec, 4, gc.TOL_FWD, gc.TOL_W)


def test_pipelined_steps_gin():
    spec = configs.small_spec(num_nodes=4000, kind="gin", dims=(16, 32, 20, 5), fanouts=(5, 4, 3),
                              batch=128, steps=4)
    _pipelined_parity(spec, 4, gc.TOL_FWD, gc.TOL_W)


def test_pipelined_steps_gat():
    spec = configs.small_spec(num_nodes=4000, kind="gat", dims=(16, 32, 20, 5), fanouts=(5, 4, 3),
                              batch=128, steps=4)
    _pipelined_parity(spec, 4, gc.TOL_FWD, gc.TOL_W)


def test_pipelined_steps_single_layer():
    # layer 1 is the output layer: its split-K logits are zeroed before its GEMM
    spec = configs.small_spec(num_nodes=3000, dims=(32, 10), fanouts=(5,), batch=50, steps=3)
    _pipelined_parity(spec, 3, gc.TOL_FWD, gc.TOL_W)


def test_pipelined_steps_bf16():
    spec = configs.small_spec(num_nodes=5000, feat_dtype="bf16", dims=(64, 32, 32, 11),
                              fanouts=(7, 5, 3), batch=200, steps=3)
    _pipelined_parity(spec, 3, gc.TOL_BF16, gc.TOL_BF16)


def test_train_model_bad_slot():
    from paper_2403_17092_amd import gnnhip
    spec = configs.small_spec(num_nodes=1000, dims=(16, 8, 4), fanouts=(3, 3), batch=16, steps=1)
    w = configs.make_workload(spec)
    csr = gc.csr_to_device(w.graph.rowptr, w.graph.col)
    tr = gnnhip.Trainer(spec.kind, spec.dims, w.weights, spec.batch, spec.fanouts, w.graph.num_nodes,
                        gnnhip.F32, gc.device())
    X = _feat_tensor(w.features)
    with pytest.raises(gnnhip.GnnError):
        tr.sample(csr, X, gc.seeds_to_device(w.seeds[0]), w.rng_key(0), 2)


def _events(n):
    rt = ctypes.CDLL("libamdhip64.so.7")
    rt.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
    out = []
    for _ in range(n):
        h = ctypes.c_void_p()
        assert rt.hipEventCreate(ctypes.byref(h)) == 0
        out.append(h.value)
    return rt, out


def test_launch_trace_of_a_training_step():
    from paper_2403_17092_amd import gnnhip
    gc.announce("launch trace")
    spec = configs.small_spec(num_nodes=3000, dims=(32, 24, 7), fanouts=(6, 4), batch=96, steps=1)
    w = configs.make_workload(spec)
    dev = gc.device()
    csr = gc.csr_to_device(w.graph.rowptr, w.graph.col)
    X = torch.as_tensor(w.features).to(dev)
    labels = torch.as_tensor(w.labels).to(dev)
    seeds = gc.seeds_to_device(w.seeds[0])
    tr = gnnhip.Trainer(spec.kind, spec.dims, w.weights, spec.batch, spec.fanouts,
                        w.graph.num_nodes, gnnhip.F32, dev)
    rt, ev = _events(2 * 64)
    t = gnnhip.Trace(ev)
    with t:
        tr.step(csr, X, labels, seeds, w.rng_key(0), spec.lr)
    torch.cuda.synchronize()
    names = t.names()
    assert t.dropped == 0
    # 2 layers: sampling (begin, 2 x (sample, scans)), layer 1 (aggregate
    # straight from the last hop's picks and the feature table, with the
    # hop's edge compaction in the same launch; gemm_fwd), layer 2's
    # aggregate, the output layer with the loss and its gradients (head),
    # layer 2's scatter, layer 1's gemm_dw, sgd
    expect = ["begin", "sample", "scans", "sample", "scans", "aggregate", "gemm_fwd",
              "aggregate", "head", "scatter", "gemm_dw", "sgd"]
    assert names == expect, names
    rt.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
    for i in range(len(names)):
        ms = ctypes.c_float()
        assert rt.hipEventElapsedTime(ctypes.byref(ms), ctypes.c_void_p(ev[2 * i]),
                                      ctypes.c_void_p(ev[2 * i + 1])) == 0
        assert 0.0 <= ms.value < 1000.0
    # filtered and over capacity: only the two aggregation launches, one recorded
    t2 = gnnhip.Trace(ev[:2], only="aggregate")
    with t2:
        tr.step(csr, X, labels, seeds, w.rng_key(0), spec.lr)
    torch.cuda.synchronize()
    assert t2.names() == ["aggregate"] and t2.dropped == 1
    assert gnnhip.check_errors() == 0


@pytest.mark.parametrize("kind,dims,fanouts", [
    ("sage_mean", (32, 24, 7), (6, 4)),          # fused output layer: gradient partials
    ("gcn", (16, 20, 20, 72), (5, 4, 3)),        # separate output layer (72 classes)
    ("gin", (32, 24, 7), (6, 4)),                # two weight matrices per layer
    ("gat", (32, 24, 7), (6, 4)),                # weights and attention vectors
])
def test_adam_steps(kind, dims, fanouts):
    # Adam as the update rule: each step's new weights and moments equal the
    # oracle's Adam applied to the gradient the step computed (read back), and
    # the first step's loss and gradient match the oracle's
    from oracle import model as omodel
    from oracle import optim
    from paper_2403_17092_amd import gnnhip
    spec = configs.small_spec(num_nodes=5000, avg_degree=10.0, kind=kind, dims=dims,
                              fanouts=fanouts, batch=48, steps=4)
    w = configs.make_workload(spec)
    dev = gc.device()
    csr = gc.csr_to_device(w.graph.rowptr, w.graph.col)
    X = torch.as_tensor(w.features).to(dev)
    labels = torch.as_tensor(w.labels).to(dev)
    tr = gnnhip.Trainer(kind, dims, w.weights, spec.batch, fanouts, w.graph.num_nodes, gnnhip.F32,
                        dev, optimizer="adam")
    lr = 0.01
    Wh = tr.weights.double().cpu().numpy()
    m = np.zeros_like(Wh)
    v = np.zeros_like(Wh)
    for s in range(4):
        gc.announce("adam step", kind, dims, s)
        loss = tr.step(csr, X, labels, gc.seeds_to_device(w.seeds[s]), w.rng_key(s), lr)
        torch.cuda.synchronize()
        assert gnnhip.check_errors() == 0
        assert tr.opt.steps == s + 1
        g = tr.inspect()["dweights"].astype(np.float64)
        if s == 0:
            ref = omodel.train_step(w.graph.rowptr, w.graph.col, w.features, w.labels, w.seeds[0],
                                    fanouts, w.rng_key(0), kind,
                                    [x.astype(np.float64) for x in w.weights], lr)
            assert abs(loss.item() - ref["loss"]) <= gc.TOL_FWD * abs(ref["loss"])
            helpers.assert_close(g, np.concatenate([x.ravel() for x in ref["dW"]]), gc.TOL_GRAD,
                                 "step 0 gradient")
        m_prev = m
        Wh, m, v = optim.adam(Wh, g, m, v, s + 1, lr)
        # the first moment sums terms of either sign: its fp32 rounding error
        # scales with the terms (beta1 |m_prev|, (1 - beta1) |g|), not with |m|
        got_m = tr.adam_m.double().cpu().numpy()
        bound = 1e-5 * np.abs(m) + 1e-6 * (0.9 * np.abs(m_prev) + 0.1 * np.abs(g)) + 1e-12
        assert np.all(np.abs(got_m - m) <= bound), np.max(np.abs(got_m - m) / bound)
        np.testing.assert_allclose(tr.adam_v.double().cpu().numpy(), v, rtol=1e-5, atol=1e-12)
        np.testing.assert_allclose(tr.weights.double().cpu().numpy(), Wh, rtol=1e-5, atol=1e-6)
        # carry the GPU's state into the next step (each step checks one step's rounding)
        Wh = tr.weights.double().cpu().numpy()
        m = got_m
        v = tr.adam_v.double().cpu().numpy()


def test_adam_pipelined_steps_match_serial():
    # the pipelined loop advances Adam's step count once per step, in order
    from paper_2403_17092_amd import gnnhip
    spec = configs.small_spec(num_nodes=5000, avg_degree=10.0, dims=(32, 24, 7), fanouts=(6, 4),
                              batch=48, steps=5)
    w = configs.make_workload(spec)
    dev = gc.device()
    csr = gc.csr_to_device(w.graph.rowptr, w.graph.col)
    X = torch.as_tensor(w.features).to(dev)
    labels = torch.as_tensor(w.labels).to(dev)
    mk = lambda: gnnhip.Trainer(spec.kind, spec.dims, w.weights, spec.batch, spec.fanouts,
                                w.graph.num_nodes, gnnhip.F32, dev, optimizer="adam")
    a, b = mk(), mk()
    batches = [(gc.seeds_to_device(w.seeds[s]), w.rng_key(s)) for s in range(5)]
    gc.announce("adam serial vs pipelined")
    for sd, k in batches:
        a.step(csr, X, labels, sd, k, 0.01)
    b.run_pipelined(csr, X, labels, batches, 0.01)
    torch.cuda.synchronize()
    assert gnnhip.check_errors() == 0
    assert a.opt.steps == b.opt.steps == 5
    helpers.assert_close(b.weights.cpu().numpy(), a.weights.cpu().numpy(), gc.TOL_W, "weights")
    helpers.assert_close(b.adam_v.cpu().numpy(), a.adam_v.cpu().numpy(), gc.TOL_GRAD, "second moment")
