"""Forward, loss, backward and SGD of one mini-batch training step (CPU oracle).

Part of the CPU oracle (test infrastructure).  float64 throughout; bfloat16
features are widened exactly.

The paper fixes (section 2.1):
  GCN layer        H_l = sigma(Ahat H_{l-1} W_l)                       eq. (1)
  GraphSAGE layer  H_l = sigma(H_{l-1} W1_l + Ahat H_{l-1} W2_l)        eq. (2)
and (section 2.2, eq. (3)) the SGD step uses the mean over the batch of the
per-root loss gradients.  It names GIN as another supported message-passing
model; GIN is taken from its definition (Xu et al., "How Powerful are Graph
Neural Networks?", ICLR 2019, eq. 4.1):
  GIN layer        H_l = sigma(MLP_l((1 + eps) H_{l-1} + sum of neighbours))
and GAT from its definition (Velickovic et al., "Graph Attention Networks",
ICLR 2018, eqs. 1-4, one attention head):
  GAT layer        T = H_{l-1} W;  e_vu = LeakyReLU(a_l . T_v + a_r . T_u);
                   alpha_v. = softmax over u in N(v) + {v} of e_vu;
                   H_l = sigma(sum_u alpha_vu T_u)
Readings where the paper is silent:

* Ahat on a sampled block (rows = dst nodes, columns = src nodes):
  - GraphSAGE-mean: row v averages v's sampled neighbours, weight 1/c_v with
    c_v the number of sampled edges of v (a row with c_v = 0 is all zero);
  - GCN: symmetric normalisation of the block with one self edge per dst
    node: weight 1/sqrt(d_out(u) d_in(v)) for every sampled edge (v, u) and
    for (v, v), where d_in(v) = c_v + 1 and d_out(u) counts the edges whose
    source is u plus one if u is itself a dst node.  On the full graph with
    every node a seed and budgets >= max degree this is Kipf & Welling's
    D^-1/2 (A + I) D^-1/2.
* GIN on a sampled block: row v sums its sampled neighbours and adds its own
  row (eps = 0, the GIN-0 variant); MLP_l is two linear layers with a ReLU
  between them, W_a [F_{l-1} x F_l] then W_b [F_l x F_l] (stored in that
  order), no bias or batch normalisation.
* GAT on a sampled block: v attends over its sampled neighbours and itself
  (the self edge the GAT paper includes), one head, LeakyReLU slope 0.2 on
  the scores; parameters W [F_{l-1} x F_l] then a [2 x F_l] (a_l, the dst
  side, then a_r, the src side).
* sigma is ReLU on every layer but the last; no bias, dropout or normalisation.
* The loss is softmax cross-entropy averaged over the batch.
* The optimiser is plain SGD: W <- W - lr dW.
* Input features are not trained, so layer 1 has no input gradient.
* Precision (the paper states none): float64 everywhere, except that a run
  whose features are stored as bfloat16 takes layer 1's GraphSAGE / GCN
  products on bfloat16 operands, as a bf16 matrix unit would: the forward
  product's inputs (the node's own rows, the aggregate, the weights) and the
  weight gradient's inputs (the same rows and the gradient of the layer's
  pre-activation) are rounded to bfloat16 (nearest, ties to even), and the
  products are summed exactly.  The weights themselves stay full precision.
"""
from __future__ import annotations

from typing import List, Optional, Sequence

import numpy as np
import scipy.sparse as sp

from . import sampling

SAGE_MEAN = "sage_mean"
GCN = "gcn"
GIN = "gin"
GAT = "gat"
GAT_SLOPE = 0.2


def widen(x: np.ndarray) -> np.ndarray:
    """float64 copy of features stored as float32, or as uint16 bfloat16 bits."""
    x = np.asarray(x)
    if x.dtype == np.uint16:
        return (x.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)
    return x.astype(np.float64)


def round_bf16(x: np.ndarray) -> np.ndarray:
    """x rounded to the nearest bfloat16 (8 significant bits, ties to even),
    as float64.  bfloat16 keeps float32's exponent range; the magnitudes here
    stay inside its normal range, where rounding the magnitude to 7 stored
    fraction bits is the whole operation."""
    x = np.ascontiguousarray(x, dtype=np.float64)
    u = x.view(np.uint64)
    drop = np.uint64(52 - 7)                     # fraction bits bfloat16 does not keep
    half = np.uint64(1) << (drop - np.uint64(1))
    odd = (u >> drop) & np.uint64(1)
    r = (u + (half - np.uint64(1)) + odd) & ~((np.uint64(1) << drop) - np.uint64(1))
    return r.view(np.float64)


def is_bf16_features(X) -> bool:
    return np.asarray(X).dtype == np.uint16


def gather(X: np.ndarray, ids: np.ndarray) -> np.ndarray:
    """Rows of the feature matrix for the given node ids (the data-fetching step)."""
    return widen(np.asarray(X)[np.asarray(ids, dtype=np.int64)])


def edge_rows(block: sampling.Block) -> np.ndarray:
    """dst index of every edge."""
    c = np.diff(block.indptr)
    return np.repeat(np.arange(block.n_dst, dtype=np.int64), c)


def out_degree(block: sampling.Block) -> np.ndarray:
    """d_out(u) = #{edges with source u} + [u is a dst node], for every src node u."""
    d = np.bincount(block.indices, minlength=block.n_src).astype(np.int64)
    d[: block.n_dst] += 1
    return d


def agg_matrix(block: sampling.Block, kind: str) -> sp.csr_matrix:
    """Ahat of the block as an explicit sparse [n_dst x n_src] matrix."""
    rows = edge_rows(block)
    cols = block.indices.astype(np.int64)
    c = np.diff(block.indptr).astype(np.float64)
    if kind == SAGE_MEAN:
        vals = 1.0 / c[rows] if rows.size else np.zeros(0)
    elif kind == GCN:
        d_out = out_degree(block).astype(np.float64)
        d_in = c + 1.0
        self_rows = np.arange(block.n_dst, dtype=np.int64)
        rows = np.concatenate([rows, self_rows])
        cols = np.concatenate([cols, self_rows])
        vals = 1.0 / np.sqrt(d_out[cols] * d_in[rows])
    elif kind == GIN:
        # sum over the sampled neighbours plus the node itself (eps = 0)
        self_rows = np.arange(block.n_dst, dtype=np.int64)
        rows = np.concatenate([rows, self_rows])
        cols = np.concatenate([cols, self_rows])
        vals = np.ones(rows.shape[0])
    else:
        raise ValueError(kind)
    return sp.csr_matrix((vals, (rows, cols)), shape=(block.n_dst, block.n_src))


def mean_aggregate(block: sampling.Block, h: np.ndarray) -> np.ndarray:
    """GraphSAGE-mean rows of Ahat h: the sum of v's sampled neighbour rows, then
    one division by c_v (0 for a row with none).  The sum of a few feature rows
    is exact in float64, so each entry is the correctly rounded mean -- the
    rounding the bfloat16 products take rests on that (a mean of bf16 values is
    often exactly halfway between two bf16 values)."""
    rows = edge_rows(block)
    S = sp.csr_matrix((np.ones(rows.shape[0]), (rows, block.indices.astype(np.int64))),
                      shape=(block.n_dst, block.n_src))
    c = np.diff(block.indptr).astype(np.float64)
    sums = S @ np.asarray(h, dtype=np.float64)
    return np.divide(sums, c[:, None], out=np.zeros_like(sums), where=c[:, None] > 0)


def relu(z):
    return np.maximum(z, 0.0)


def gat_edges(block: sampling.Block):
    """(dst, src) of every edge a GAT layer attends over: the sampled edges,
    then one self edge per dst node."""
    self_rows = np.arange(block.n_dst, dtype=np.int64)
    rows = np.concatenate([edge_rows(block), self_rows])
    cols = np.concatenate([np.asarray(block.indices, dtype=np.int64), self_rows])
    return rows, cols


def gat_forward(block: sampling.Block, h: np.ndarray, W: np.ndarray, a: np.ndarray):
    """One GAT layer before its activation: returns (out [n_dst x F_out], cache)."""
    rows, cols = gat_edges(block)
    T = h @ W
    pre = (T[: block.n_dst] @ a[0])[rows] + (T @ a[1])[cols]
    e = np.where(pre > 0, pre, GAT_SLOPE * pre)
    # softmax over each dst row's edges
    m = np.full(block.n_dst, -np.inf)
    np.maximum.at(m, rows, e)
    ex = np.exp(e - m[rows])
    alpha = ex / np.bincount(rows, weights=ex, minlength=block.n_dst)[rows]
    Aat = sp.csr_matrix((alpha, (rows, cols)), shape=(block.n_dst, block.n_src))
    return Aat @ T, dict(rows=rows, cols=cols, T=T, pre=pre, alpha=alpha, Aat=Aat)


def gat_backward(block: sampling.Block, h: np.ndarray, W: np.ndarray, a: np.ndarray, c: dict,
                 dout: np.ndarray):
    """Gradients of one GAT layer from dout = dLoss/d(out): (dW, da, dh)."""
    rows, cols, T, alpha = c["rows"], c["cols"], c["T"], c["alpha"]
    dT = c["Aat"].T @ dout                                  # through out = alpha T
    dalpha = np.sum(dout[rows] * T[cols], axis=1)
    # softmax: de_vu = alpha_vu (dalpha_vu - sum_w alpha_vw dalpha_vw)
    s = np.bincount(rows, weights=alpha * dalpha, minlength=block.n_dst)
    de = alpha * (dalpha - s[rows])
    dpre = de * np.where(c["pre"] > 0, 1.0, GAT_SLOPE)
    ds_l = np.bincount(rows, weights=dpre, minlength=block.n_dst)
    ds_r = np.bincount(cols, weights=dpre, minlength=block.n_src)
    da = np.stack([T[: block.n_dst].T @ ds_l, T.T @ ds_r])
    dT[: block.n_dst] += np.outer(ds_l, a[0])
    dT += np.outer(ds_r, a[1])
    return h.T @ dT, da, dT @ W.T


def layer_weights(kind: str, weights: Sequence[np.ndarray], layer: int):
    """Weights of layer `layer` (1-based) from the flat list."""
    if kind in (SAGE_MEAN, GIN, GAT):
        return weights[2 * (layer - 1)], weights[2 * (layer - 1) + 1]
    return (weights[layer - 1],)


def softmax_xent(logits: np.ndarray, y: np.ndarray):
    """Mean softmax cross-entropy over the rows and its gradient w.r.t. the logits."""
    b = logits.shape[0]
    m = logits.max(axis=1, keepdims=True)
    e = np.exp(logits - m)
    s = e.sum(axis=1, keepdims=True)
    logp = logits - m - np.log(s)
    loss = -logp[np.arange(b), y].mean() if b else 0.0
    p = e / s
    d = p.copy()
    d[np.arange(b), y] -= 1.0
    return float(loss), d / max(b, 1)


def run_model(kind: str, weights: Sequence[np.ndarray], layer_blocks: List[sampling.Block],
              H0: np.ndarray, y: np.ndarray, lr: float, readout: Optional[np.ndarray] = None,
              bf16_layer1: bool = False):
    """Forward, loss, backward and SGD.  layer_blocks[l-1] is the block layer l runs on;
    H0 has one row per src node of layer 1's block.  `readout` selects the rows of the
    last layer's output that carry a label (default: all of them).  bf16_layer1: layer
    1's GraphSAGE / GCN products take bfloat16-rounded operands (see the module note)."""
    L = len(layer_blocks)
    # operand rounding of a layer's products: bfloat16 on layer 1 if asked
    def q(l, x):
        return round_bf16(x) if (bf16_layer1 and l == 1 and kind in (SAGE_MEAN, GCN)) else x

    W = [np.asarray(w, dtype=np.float64) for w in weights]
    A = [None if kind == GAT else agg_matrix(b, kind) for b in layer_blocks]
    H = [np.asarray(H0, dtype=np.float64)]
    aggs, Zs, Ps, gat = [], [], [], []
    for l in range(1, L + 1):
        blk, h = layer_blocks[l - 1], H[l - 1]
        ws = layer_weights(kind, W, l)
        if kind == GAT:
            # the attention-weighted sum is the layer's aggregate and its pre-activation
            z, cache = gat_forward(blk, h, ws[0], ws[1])
            gat.append(cache)
            aggs.append(z)
            Zs.append(z)
            H.append(relu(z) if l < L else z)
            continue
        agg = mean_aggregate(blk, h) if kind == SAGE_MEAN else A[l - 1] @ h
        if kind == SAGE_MEAN:
            z = q(l, h[: blk.n_dst]) @ q(l, ws[0]) + q(l, agg) @ q(l, ws[1])
        elif kind == GIN:
            p_ = agg @ ws[0]          # the MLP's first linear layer
            Ps.append(p_)
            z = relu(p_) @ ws[1]
        else:
            z = q(l, agg) @ q(l, ws[0])
        aggs.append(agg)
        Zs.append(z)
        H.append(relu(z) if l < L else z)
    out = H[L]
    logits = out if readout is None else out[np.asarray(readout, dtype=np.int64)]
    loss, dlogits = softmax_xent(logits, np.asarray(y, dtype=np.int64))
    dZ = np.zeros_like(out)
    if readout is None:
        dZ = dlogits
    else:
        np.add.at(dZ, np.asarray(readout, dtype=np.int64), dlogits)

    dW = [None] * len(W)
    dHs = [None] * (L + 1)
    for l in range(L, 0, -1):
        blk, h = layer_blocks[l - 1], H[l - 1]
        ws = layer_weights(kind, W, l)
        if kind == GAT:
            dW[2 * (l - 1)], dW[2 * (l - 1) + 1], dH = gat_backward(blk, h, ws[0], ws[1],
                                                                  gat[l - 1], dZ)
            if l == 1:
                break
            dHs[l - 1] = dH
            dZ = dH * (Zs[l - 2] > 0)
            continue
        if kind == SAGE_MEAN:
            dW[2 * (l - 1)] = q(l, h[: blk.n_dst]).T @ q(l, dZ)
            dW[2 * (l - 1) + 1] = q(l, aggs[l - 1]).T @ q(l, dZ)
        elif kind == GIN:
            m_ = relu(Ps[l - 1])
            dW[2 * (l - 1) + 1] = m_.T @ dZ
            dP = (dZ @ ws[1].T) * (Ps[l - 1] > 0)
            dW[2 * (l - 1)] = aggs[l - 1].T @ dP
        else:
            dW[l - 1] = q(l, aggs[l - 1]).T @ q(l, dZ)
        if l == 1:
            break
        if kind == SAGE_MEAN:
            dH = A[l - 1].T @ (dZ @ ws[1].T)
            dH[: blk.n_dst] += dZ @ ws[0].T
        elif kind == GIN:
            dH = A[l - 1].T @ (dP @ ws[0].T)
        else:
            dH = A[l - 1].T @ (dZ @ ws[0].T)
        dHs[l - 1] = dH
        dZ = dH * (Zs[l - 2] > 0)
    W_new = [w - lr * g for w, g in zip(W, dW)]
    return dict(agg=aggs, Z=Zs, H=H, logits=logits, loss=loss, dW=dW, W_new=W_new, dH=dHs,
                dlogits=dlogits, P=Ps, att=[c["alpha"] for c in gat])


def train_step(rowptr, col, X, labels, seeds, fanouts, rng_key: int, kind: str,
               weights: Sequence[np.ndarray], lr: float):
    """One neighbour-sampled training step: sample, gather, forward, loss, backward, SGD.
    Features stored as bfloat16 (uint16 bits) select the bfloat16 layer-1 products."""
    blocks = sampling.sample_blocks(rowptr, col, seeds, fanouts, rng_key)
    xg = gather(X, blocks[-1].src_nodes)
    y = np.asarray(labels)[np.asarray(seeds, dtype=np.int64)]
    res = run_model(kind, weights, blocks[::-1], xg, y, lr, bf16_layer1=is_bf16_features(X))
    res["blocks"] = blocks
    res["xg"] = xg
    return res
