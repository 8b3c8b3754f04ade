"""Pins for the oracle's bfloat16 layer-1 products (no GPU): the rounding
itself, and the forward and weight-gradient products of layer 1 against what
the arithmetic fixes -- exact when every operand is already a bfloat16 value,
and otherwise within the unit-roundoff bound of two rounded factors."""
import numpy as np
import pytest
import torch

from oracle import model, sampling
from tests import helpers

U = 2.0 ** -8   # unit roundoff of bfloat16 (8 significant bits, round to nearest)


def test_round_bf16_hand_cases():
    one = 1.0
    cases = [
        (one + 2.0 ** -8, one),                        # tie between 1 and 1 + 2^-7: to even
        (one + 3 * 2.0 ** -8, one + 2.0 ** -6),        # tie between 1 + 2^-7 and 1 + 2^-6: to even
        (one + 2.0 ** -8 + 2.0 ** -30, one + 2.0 ** -7),  # above the tie: up
        (one + 2.0 ** -8 - 2.0 ** -30, one),           # below the tie: down
        (-(one + 3 * 2.0 ** -8), -(one + 2.0 ** -6)),  # sign kept, magnitude rounded
        (0.0, 0.0), (1.5, 1.5), (-0.0078125, -0.0078125), (3.0 * 2.0 ** -20, 3.0 * 2.0 ** -20),
        (255.0, 255.0), (257.0, 256.0), (259.0, 260.0),  # integers past 2^8: spacing 2
    ]
    x = np.array([c[0] for c in cases])
    want = np.array([c[1] for c in cases])
    got = model.round_bf16(x)
    assert np.array_equal(got, want), (got, want)
    assert np.array_equal(np.signbit(got), np.signbit(want))


def test_round_bf16_equals_torch_conversion_of_float32():
    g = np.random.Generator(np.random.PCG64(5))
    x32 = (g.normal(size=200_000) * np.exp(g.uniform(-30, 30, size=200_000))).astype(np.float32)
    # exact ties in the low 16 bits, with an even and an odd kept last bit
    bits = g.integers(0x3000_0000, 0x4800_0000, size=20_000, dtype=np.uint32)
    ties = ((bits & np.uint32(0xFFFF0000)) | np.uint32(0x8000)).view(np.float32)
    x32 = np.concatenate([x32, ties, -ties])
    want = torch.from_numpy(x32).to(torch.bfloat16).to(torch.float64).numpy()
    got = model.round_bf16(x32.astype(np.float64))
    assert np.array_equal(got, want)
    assert np.array_equal(model.round_bf16(got), got)  # idempotent


def _one_pick_instance(kind, seed):
    """A 2-layer step whose layer-1 aggregate is bf16-exact: budget 1 per hop
    (SAGE-mean of one row is that row) and bf16-valued features and weights."""
    rowptr, col = helpers.random_graph(60, 0.1, seed)
    deg = np.diff(rowptr)
    seeds = np.flatnonzero(deg > 0)[:12].astype(np.int32)
    blocks = sampling.sample_blocks(rowptr, col, seeds, [1, 1], 7)
    g = np.random.Generator(np.random.PCG64(seed))
    X = model.round_bf16(g.normal(size=(60, 8)))
    dims = (8, 6, 3)
    ws = []
    for l in range(1, 3):
        for _ in range(2 if kind == model.SAGE_MEAN else 1):
            ws.append(model.round_bf16(g.normal(0, 0.5, (dims[l - 1], dims[l]))))
    y = g.integers(0, 3, size=len(seeds))
    return blocks, X[blocks[-1].src_nodes], y, ws


def test_bf16_layer1_forward_exact_on_bf16_operands():
    blocks, H0, y, ws = _one_pick_instance(model.SAGE_MEAN, 3)
    a = model.run_model(model.SAGE_MEAN, ws, blocks[::-1], H0, y, 0.0, bf16_layer1=True)
    b = model.run_model(model.SAGE_MEAN, ws, blocks[::-1], H0, y, 0.0, bf16_layer1=False)
    for za, zb in zip(a["Z"], b["Z"]):
        assert np.allclose(za, zb, rtol=0, atol=1e-13)
    assert abs(a["loss"] - b["loss"]) <= 1e-13


@pytest.mark.parametrize("kind", [model.SAGE_MEAN, model.GCN])
def test_bf16_layer1_products_within_rounding_bound(kind):
    g = np.random.Generator(np.random.PCG64(11))
    rowptr, col = helpers.random_graph(80, 0.12, 4)
    seeds = np.arange(0, 80, 5, dtype=np.int32)
    blocks = sampling.sample_blocks(rowptr, col, seeds, [4, 3], 9)
    X = model.round_bf16(g.normal(size=(80, 10)))
    H0 = X[blocks[-1].src_nodes]
    dims = (10, 12, 4)
    ws = []
    for l in range(1, 3):
        for _ in range(2 if kind == model.SAGE_MEAN else 1):
            ws.append(g.normal(0, 0.4, (dims[l - 1], dims[l])))
    y = g.integers(0, 4, size=len(seeds))
    r = model.run_model(kind, ws, blocks[::-1], H0, y, 0.0, bf16_layer1=True)
    blk = blocks[-1]
    agg = r["agg"][0]
    parts = [(H0[: blk.n_dst], 0), (agg, 1)] if kind == model.SAGE_MEAN else [(agg, 0)]
    bound = 2 * U + U * U
    # forward: Z1 = sum of products of two rounded factors
    z_exact = sum(x @ ws[i] for x, i in parts)
    z_abs = sum(np.abs(x) @ np.abs(ws[i]) for x, i in parts)
    err = np.abs(r["Z"][0] - z_exact)
    assert (err <= bound * z_abs + 1e-12).all()
    assert err.max() > 0  # the operands were rounded
    # weight gradient: dW1 = rows^T dZ1 with both factors rounded, dZ1 the
    # run's own pre-activation gradient of layer 1
    dZ1 = r["dH"][1] * (r["Z"][0] > 0)
    for x, i in parts:
        exact = x.T @ dZ1
        e = np.abs(r["dW"][i] - exact)
        assert (e <= bound * (np.abs(x).T @ np.abs(dZ1)) + 1e-15).all()
        assert e.max() > 0
    # only layer 1 takes the rounding: layer 2's weight gradient is H1^T dZ2 exactly
    k = 2 if kind == model.SAGE_MEAN else 1
    dZ2 = r["dlogits"]
    if kind == model.SAGE_MEAN:
        exact2 = r["agg"][1].T @ dZ2
        assert np.allclose(r["dW"][k + 1], exact2, rtol=0, atol=1e-14)
    else:
        assert np.allclose(r["dW"][k], r["agg"][1].T @ dZ2, rtol=0, atol=1e-14)


def test_bf16_features_select_bf16_products():
    from workloads import configs
    spec = configs.small_spec(num_nodes=800, feat_dtype="bf16", dims=(16, 8, 4), fanouts=(4, 3),
                              batch=32)
    w = configs.make_workload(spec)
    a = model.train_step(w.graph.rowptr, w.graph.col, w.features, w.labels, w.seeds[0], spec.fanouts,
                         1, spec.kind, w.weights, spec.lr)
    blocks = a["blocks"]
    H0 = model.gather(w.features, blocks[-1].src_nodes)
    y = np.asarray(w.labels)[w.seeds[0]]
    b = model.run_model(spec.kind, w.weights, blocks[::-1], H0, y, spec.lr, bf16_layer1=True)
    c = model.run_model(spec.kind, w.weights, blocks[::-1], H0, y, spec.lr, bf16_layer1=False)
    assert all(np.array_equal(x, z) for x, z in zip(a["dW"], b["dW"]))
    assert not np.array_equal(a["dW"][1], c["dW"][1])


def test_bf16_rounds_the_output_gradient():
    # rows and weights already bf16 values: only dZ1's rounding moves dW1,
    # by at most one unit roundoff of each product
    blocks, H0, y, ws = _one_pick_instance(model.SAGE_MEAN, 8)
    r = model.run_model(model.SAGE_MEAN, ws, blocks[::-1], H0, y, 0.0, bf16_layer1=True)
    dZ1 = r["dH"][1] * (r["Z"][0] > 0)
    agg = r["agg"][0]
    assert np.array_equal(model.round_bf16(agg), agg)
    e = np.abs(r["dW"][1] - agg.T @ dZ1)
    assert e.max() > 0
    assert (e <= U * (np.abs(agg).T @ np.abs(dZ1)) + 1e-15).all()


def test_bf16_rounds_the_weights():
    # bf16 rows with full-precision weights: only the weights' rounding moves Z1
    blocks, H0, y, ws = _one_pick_instance(model.SAGE_MEAN, 9)
    g = np.random.Generator(np.random.PCG64(2))
    ws = [w + g.normal(0, 1e-3, w.shape) for w in ws]
    r = model.run_model(model.SAGE_MEAN, ws, blocks[::-1], H0, y, 0.0, bf16_layer1=True)
    n = blocks[-1].n_dst
    exact = H0[:n] @ ws[0] + r["agg"][0] @ ws[1]
    e = np.abs(r["Z"][0] - exact)
    assert e.max() > 0
    assert (e <= U * (np.abs(H0[:n]) @ np.abs(ws[0]) + np.abs(r["agg"][0]) @ np.abs(ws[1])) + 1e-13).all()


def _bf16_rne_exact(q):
    """Round the rational q to the nearest bfloat16 (ties to even), exactly."""
    from fractions import Fraction
    if q == 0:
        return Fraction(0)
    sign = -1 if q < 0 else 1
    a = abs(q)
    e = 0
    while a >= 2:
        a /= 2
        e += 1
    while a < 1:
        a *= 2
        e -= 1
    scaled = a * 128                   # 8 significant bits: 1.xxxxxxx
    n = int(scaled)
    rem = scaled - n
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and n % 2 == 1):
        n += 1
    return sign * Fraction(n, 128) * Fraction(2) ** e


def test_mean_aggregate_rounds_like_the_exact_mean():
    # means of bf16 values land exactly halfway between bf16 values; the oracle's
    # aggregate must round, as the exact mean does, to the even neighbour
    from fractions import Fraction
    g = np.random.Generator(np.random.PCG64(21))
    n, f = 400, 16
    rowptr, col = helpers.random_graph(n, 0.03, 6)
    X = model.round_bf16(g.normal(size=(n, f)))
    seeds = np.arange(0, n, 3, dtype=np.int32)
    blk = sampling.sample_blocks(rowptr, col, seeds, [5], 2)[0]
    h = X[blk.src_nodes]
    agg = model.mean_aggregate(blk, h)
    got = model.round_bf16(agg)
    ties = 0
    for v in range(blk.n_dst):
        e0, e1 = blk.indptr[v], blk.indptr[v + 1]
        c = e1 - e0
        for j in range(f):
            if c == 0:
                assert got[v, j] == 0.0
                continue
            exact = sum(Fraction(float(h[u, j])) for u in blk.indices[e0:e1]) / c
            want = _bf16_rne_exact(exact)
            assert Fraction(float(got[v, j])) == want, (v, j, float(exact), float(want), got[v, j])
            lo = _bf16_rne_exact(exact - Fraction(1, 2 ** 40))
            ties += int(lo != want)
    assert ties > 0  # the instance does hit rounding boundaries
