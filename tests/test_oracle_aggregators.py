"""Pins for the oracle's aggregator variants (gamma = mean and gamma = max, the
compared variants of Sec. 4) and Algorithm 2's output dense layers
(z = G2 ReLU(G1 h + g)).

Aggregators: with Q = I, q = 0 and non-negative inputs the transformed rows are
the inputs themselves, and W = [0 | I] keeps only the pooled vector, so a layer
reduces to the normalised numpy mean / element-wise max of the neighbour rows.
Further: a single neighbour or identical neighbours make the three aggregators
agree; mean and max ignore the neighbours' order and weights; an empty
neighbourhood pools to zero; the layer-wise and Algorithm 2 routes agree.

Output layers: a hand-worked 2-D example, identity and single-entry matrices
that expose a transposed G1 or G2, a bias-only case and linearity in G2.
"""

import numpy as np
import pytest

import synth


def _nbrs(rng, n_out, n_src, T, allow_empty=True):
    idx = np.full((n_out, T), -1, np.int32)
    wts = np.zeros((n_out, T), np.float32)
    for r in range(n_out):
        k = int(rng.integers(0 if allow_empty else 1, T + 1))
        if k:
            idx[r, :k] = rng.choice(n_src, k, replace=False)
            c = rng.integers(1, 9, size=k).astype(np.float32)
            wts[r, :k] = c / np.float32(c.sum())
    return idx, wts


def _select_pooled(d):
    return np.concatenate([np.zeros((d, d)), np.eye(d)], axis=1)


@pytest.mark.parametrize("pool,reduce", [("mean", np.mean), ("max", np.max)])
def test_identity_transform_reduces_to_numpy(orc, pool, reduce):
    rng = np.random.default_rng(4)
    n, d, T = 50, 7, 6
    h = np.abs(rng.standard_normal((n, d)))
    idx, wts = _nbrs(rng, n, n, T, allow_empty=False)
    out = orc.convolve_layer(h, n, np.eye(d), np.zeros(d), _select_pooled(d), np.zeros(d), idx,
                             wts, pool=pool)
    for r in range(n):
        v = reduce(h[idx[r][idx[r] >= 0]], axis=0)
        np.testing.assert_allclose(out[r], v / np.linalg.norm(v), rtol=1e-12, atol=1e-14)


def test_single_or_identical_neighbours_make_the_aggregators_agree(orc):
    rng = np.random.default_rng(5)
    n, d_in, m, d_out, T = 30, 6, 5, 4, 4
    h = rng.standard_normal((n, d_in))
    wl = synth.Workload("t", 1, 1, "uniform8", 0, 8, None, d_in, m, d_out, 1, 1, 1, T, "f32", 6)
    L = synth.make_layers(wl)[0]
    # Row r: one neighbour (weight 1), or the same neighbour repeated is not a
    # valid table (ids are distinct), so identical rows come from duplicated
    # feature rows: nodes r and r + n share one feature vector.
    idx = np.full((n, T), -1, np.int32)
    wts = np.zeros((n, T), np.float32)
    idx[:, 0] = rng.integers(0, n, size=n)
    wts[:, 0] = 1.0
    outs = [orc.convolve_layer(h, n, L["Q"], L["q"], L["W"], L["w"], idx, wts, pool=p)
            for p in ("importance", "mean", "max")]
    np.testing.assert_allclose(outs[1], outs[0], rtol=1e-13, atol=1e-15)
    np.testing.assert_allclose(outs[2], outs[0], rtol=1e-13, atol=1e-15)
    h2 = np.concatenate([h, h])
    idx2 = np.stack([idx[:, 0], idx[:, 0] + n, -np.ones(n, np.int32), -np.ones(n, np.int32)], 1)
    wts2 = np.zeros((n, T), np.float32)
    wts2[:, :2] = 0.5
    outs2 = [orc.convolve_layer(h2, 2 * n, L["Q"], L["q"], L["W"], L["w"], idx2.astype(np.int32),
                                wts2, pool=p) for p in ("importance", "mean", "max")]
    for o in outs2:
        np.testing.assert_allclose(o, outs[0], rtol=1e-12, atol=1e-14)


@pytest.mark.parametrize("pool", ["mean", "max"])
def test_order_and_weights_do_not_matter(orc, pool):
    rng = np.random.default_rng(6)
    n, d_in, m, d_out, T = 40, 8, 6, 5, 7
    h = rng.standard_normal((n, d_in))
    wl = synth.Workload("t", 1, 1, "uniform8", 0, 8, None, d_in, m, d_out, 1, 1, 1, T, "f32", 7)
    L = synth.make_layers(wl)[0]
    idx, wts = _nbrs(rng, n, n, T)
    a = orc.convolve_layer(h, n, L["Q"], L["q"], L["W"], L["w"], idx, wts, pool=pool)
    perm = rng.permutation(T)
    idx_p = idx[:, perm]
    wts_p = rng.random((n, T)).astype(np.float32)  # any weights
    b = orc.convolve_layer(h, n, L["Q"], L["q"], L["W"], L["w"], idx_p, wts_p, pool=pool)
    np.testing.assert_allclose(b, a, rtol=1e-12, atol=1e-14)


@pytest.mark.parametrize("pool", ["importance", "mean", "max"])
def test_empty_neighbourhood_pools_to_zero(orc, pool):
    rng = np.random.default_rng(7)
    n, d_in, m, d_out, T = 12, 5, 4, 6, 3
    h = rng.standard_normal((n, d_in))
    wl = synth.Workload("t", 1, 1, "uniform8", 0, 8, None, d_in, m, d_out, 1, 1, 1, T, "f32", 8)
    L = synth.make_layers(wl)[0]
    idx = np.full((n, T), -1, np.int32)
    wts = np.zeros((n, T), np.float32)
    out = orc.convolve_layer(h, n, L["Q"], L["q"], L["W"], L["w"], idx, wts, pool=pool)
    z = np.maximum(h @ L["W"][:, :d_in].T + L["w"], 0.0)  # the self half only
    norm = np.linalg.norm(z, axis=1, keepdims=True)
    np.testing.assert_allclose(out, np.where(norm > 0, z / np.where(norm > 0, norm, 1), 0),
                               rtol=1e-12, atol=1e-14)


@pytest.mark.parametrize("pool", ["mean", "max"])
def test_layerwise_equals_minibatch(orc, pool):
    wl = synth.WORKLOADS["tiny"]
    data = synth.make_workload(wl)
    idx, cnt, wts, _ = orc.build_neighborhoods(data["offsets"], data["col"], wl.num_pins,
                                               wl.seed, wl.walks, wl.hops, wl.T)
    layers = [dict(L, pool=pool) for L in data["layers"]]
    full = orc.embed_all(data["x"], wl.num_pins, layers, idx, wts)
    targets = np.array([0, 17, 1999, 2000, 2499, 640], np.int32)
    mb = orc.minibatch_embed(targets, data["x"], layers, idx, wts)
    np.testing.assert_allclose(mb, full[targets], rtol=1e-12, atol=1e-14)


def test_output_mlp_worked_example(orc):
    # G1 h + g = [1 - 2 + 0.5, 2 + 2 - 1] = [-0.5, 3]; ReLU -> [0, 3];
    # G2 [0, 3] = [2*3, 0.5*3, 0*3] = [6, 1.5, 0].
    h = np.array([[1.0, -2.0]])
    G1 = np.array([[1.0, 1.0], [2.0, -1.0]])
    g = np.array([0.5, -1.0])
    G2 = np.array([[1.0, 2.0], [-1.0, 0.5], [3.0, 0.0]])
    np.testing.assert_allclose(orc.output_mlp(h, G1, g, G2), [[6.0, 1.5, 0.0]], rtol=0, atol=0)


def test_output_mlp_identity_and_transposes(orc):
    rng = np.random.default_rng(9)
    n, d_in, d_hidden, d_out = 20, 5, 7, 3
    h = rng.standard_normal((n, d_in))
    z = orc.output_mlp(h, np.eye(d_in), np.zeros(d_in), np.eye(d_in))
    np.testing.assert_allclose(z, np.maximum(h, 0.0), rtol=0, atol=0)
    # One entry each: G1[i, j] = 1 routes h_j to hidden unit i; G2[o, i] = 1
    # routes hidden unit i to output o; every other output is zero.
    i, j, o = 4, 2, 1
    G1 = np.zeros((d_hidden, d_in)); G1[i, j] = 1.0
    G2 = np.zeros((d_out, d_hidden)); G2[o, i] = 1.0
    z = orc.output_mlp(h, G1, np.zeros(d_hidden), G2)
    want = np.zeros((n, d_out)); want[:, o] = np.maximum(h[:, j], 0.0)
    np.testing.assert_allclose(z, want, rtol=0, atol=0)
    # Bias only: G1 = 0 gives ReLU(g) in every row.
    g = rng.standard_normal(d_hidden)
    G2 = rng.standard_normal((d_out, d_hidden))
    z = orc.output_mlp(h, np.zeros((d_hidden, d_in)), g, G2)
    np.testing.assert_allclose(z, np.tile(G2 @ np.maximum(g, 0.0), (n, 1)), rtol=1e-13, atol=1e-14)


def test_output_mlp_is_linear_in_G2(orc):
    rng = np.random.default_rng(10)
    n, d_in, d_hidden, d_out = 15, 6, 9, 4
    h = rng.standard_normal((n, d_in))
    G1, g = rng.standard_normal((d_hidden, d_in)), rng.standard_normal(d_hidden)
    A, B = rng.standard_normal((d_out, d_hidden)), rng.standard_normal((d_out, d_hidden))
    za, zb = orc.output_mlp(h, G1, g, A), orc.output_mlp(h, G1, g, B)
    np.testing.assert_allclose(orc.output_mlp(h, G1, g, A + 2.0 * B), za + 2.0 * zb, rtol=1e-12,
                               atol=1e-12)
