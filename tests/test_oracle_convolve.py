"""Pins for the oracle's CONVOLVE (Algorithm 1), layer-wise driver (Sec. 3.4),
MINIBATCH (Algorithm 2) and max-margin loss (Eq. 1).

Each check is a special case or invariant that a plausible slip (dropped bias,
swapped concat halves, transposed Q or W, wrong weight normalisation, missing
ReLU or norm) fails: a hand-worked example, identity / constant parameters that
reduce the layer to a plain mean or a plain normalisation, single-entry
matrices that expose a transpose, unit norms, relabelling equivariance, and the
agreement of two different dataflows (layer-wise vs Algorithm 2).
"""

import json
import os

import numpy as np
import pytest

import synth

HERE = os.path.dirname(os.path.abspath(__file__))


def test_worked_example(orc):
    with open(os.path.join(HERE, "golden", "convolve_worked_example.json")) as f:
        ex = json.load(f)
    out = orc.convolve_layer(np.array(ex["h_in"], float), ex["n_transform"], np.array(ex["Q"]),
                             np.array(ex["q"]), np.array(ex["W"]), np.array(ex["w"]),
                             np.array(ex["idx"]), np.array(ex["weights"], np.float32))
    np.testing.assert_allclose(out, np.array(ex["expected"]), rtol=0, atol=1e-15)


def _random_nbr(rng, n_out, n_transform, T, fill=0.8):
    idx = np.full((n_out, T), -1, np.int32)
    wts = np.zeros((n_out, T), np.float32)
    for r in range(n_out):
        k = int(rng.integers(0, T + 1)) if rng.random() < fill else 0
        if k:
            idx[r, :k] = rng.choice(n_transform, k, replace=False)
            c = rng.integers(1, 9, size=k).astype(np.float32)
            wts[r, :k] = c / np.float32(c.sum())
    return idx, wts


def test_identity_transform_gives_plain_mean(orc):
    rng = np.random.default_rng(1)
    n, d, T = 40, 8, 5
    h = np.abs(rng.standard_normal((n, d)))  # non-negative, so ReLU(I h) = h
    idx = np.stack([rng.choice(n, T, replace=False) for _ in range(n)]).astype(np.int32)
    wts = np.full((n, T), np.float32(1.0 / T), np.float32)
    W = np.concatenate([np.zeros((d, d)), np.eye(d)], axis=1)  # keep only n_u
    out = orc.convolve_layer(h, n, np.eye(d), np.zeros(d), W, np.zeros(d), idx, wts)
    mean = h[idx].mean(axis=1) * (np.float64(np.float32(1.0 / T)) * T)
    want = mean / np.linalg.norm(mean, axis=1, keepdims=True)
    np.testing.assert_allclose(out, want, rtol=1e-12, atol=1e-14)


def test_self_half_and_neighbour_half(orc):
    rng = np.random.default_rng(2)
    n, d, m, T = 30, 6, 4, 3
    h = rng.standard_normal((n, d))
    idx, wts = _random_nbr(rng, n, n, T, fill=1.0)
    Q = rng.standard_normal((m, d))
    # W = [I | 0]: output is normalize(ReLU(h_u)).
    W = np.concatenate([np.eye(d), np.zeros((d, m))], axis=1)
    out = orc.convolve_layer(h, n, Q, np.zeros(m), W, np.zeros(d), idx, wts)
    z = np.maximum(h, 0)
    nz = np.linalg.norm(z, axis=1, keepdims=True)
    want = np.where(nz > 0, z / np.where(nz > 0, nz, 1), 0)
    np.testing.assert_allclose(out, want, rtol=1e-13, atol=1e-15)


def test_constant_bias_paths(orc):
    rng = np.random.default_rng(3)
    n, d, m, T = 25, 5, 7, 4
    h = rng.standard_normal((n, d))
    idx, wts = _random_nbr(rng, n, n, T, fill=0.7)
    # Q = 0, q = c: every transformed neighbour is c*1, so n_u = c*sum(alpha) = c*1.
    W = np.concatenate([np.zeros((m, d)), np.eye(m)], axis=1)
    out = orc.convolve_layer(h, n, np.zeros((m, d)), np.full(m, 0.5), W, np.zeros(m), idx, wts)
    live = idx[:, 0] >= 0
    np.testing.assert_allclose(out[live], 1.0 / np.sqrt(m), rtol=1e-7)  # alpha sums to 1 in fp32
    assert np.all(out[~live] == 0)
    # W = 0, w = c: every output row is c*1 normalised.
    out = orc.convolve_layer(h, n, rng.standard_normal((m, d)), np.zeros(m), np.zeros((d, d + m)),
                             np.full(d, 0.25), idx, wts)
    np.testing.assert_allclose(out, 1.0 / np.sqrt(d), rtol=1e-14)


def test_single_entry_matrices_expose_transposes(orc):
    # One neighbour with weight 1; Q has a single 1 at (i=2, j=0) so
    # P_v[2] = ReLU(h_v[0]); W has a single 1 at (o=1, column d+2) so the output
    # is e_1 when h_v[0] > 0. A transposed Q or W lands on another coordinate.
    d, m = 3, 4
    h = np.array([[0.7, -2.0, 5.0], [1.5, 0.3, -0.2]])
    idx = np.array([[1], [0]], np.int32)
    wts = np.ones((2, 1), np.float32)
    Q = np.zeros((m, d)); Q[2, 0] = 1.0
    W = np.zeros((d, d + m)); W[1, d + 2] = 1.0
    out = orc.convolve_layer(h, 2, Q, np.zeros(m), W, np.zeros(d), idx, wts)
    np.testing.assert_array_equal(out, np.array([[0, 1, 0], [0, 1, 0]], float))
    # Row 1 pools node 0, whose h[0] < 0 is cut by ReLU: the row becomes zero.
    h2 = h.copy(); h2[0, 0] = -1.0
    out = orc.convolve_layer(h2, 2, Q, np.zeros(m), W, np.zeros(d), idx, wts)
    np.testing.assert_array_equal(out[1], np.zeros(d))


def test_unit_norm_and_relabelling(orc):
    rng = np.random.default_rng(4)
    n_pins, n, d, m, T = 50, 70, 16, 24, 6
    h = rng.standard_normal((n, d))
    idx, wts = _random_nbr(rng, n, n_pins, T, fill=0.9)
    Q, q = rng.standard_normal((m, d)) * 0.3, rng.uniform(-0.1, 0.1, m)
    W, w = rng.standard_normal((12, d + m)) * 0.3, rng.uniform(-0.1, 0.1, 12)
    out = orc.convolve_layer(h, n_pins, Q, q, W, w, idx, wts)
    norms = np.linalg.norm(out, axis=1)
    assert np.all((np.abs(norms - 1) < 1e-12) | (norms == 0))
    # Relabel pins among pins and boards among boards; outputs permute exactly.
    perm = np.concatenate([rng.permutation(n_pins), n_pins + rng.permutation(n - n_pins)])
    inv = np.argsort(perm)  # new id of old node i is inv[i]
    h_new = h[perm]
    idx_new = np.where(idx >= 0, inv[np.maximum(idx, 0)], -1).astype(np.int32)[perm]
    out_new = orc.convolve_layer(h_new, n_pins, Q, q, W, w, idx_new, wts[perm])
    np.testing.assert_array_equal(out_new, out[perm])


def test_self_rows_select_the_self_vector(orc):
    rng = np.random.default_rng(5)
    n, d, m, T = 20, 4, 6, 3
    h = rng.standard_normal((n, d))
    idx, wts = _random_nbr(rng, n, n, T)
    Q, q = rng.standard_normal((m, d)), rng.uniform(-0.1, 0.1, m)
    W, w = rng.standard_normal((5, d + m)), rng.uniform(-0.1, 0.1, 5)
    full = orc.convolve_layer(h, n, Q, q, W, w, idx, wts)
    rows = np.array([7, 0, 19, 7], np.int64)
    sub = orc.convolve_layer(h, n, Q, q, W, w, idx[rows], wts[rows], self_rows=rows)
    np.testing.assert_array_equal(sub, full[rows])


def test_minibatch_sets_brute_force(orc):
    rng = np.random.default_rng(6)
    N, T, K = 200, 5, 2
    nbr = np.full((N, T), -1, np.int32)
    for u in range(N):
        k = int(rng.integers(0, T + 1))
        nbr[u, :k] = rng.choice(N, k, replace=False)
    targets = rng.choice(N, 12, replace=False).astype(np.int32)
    sets = orc.minibatch_sets(targets, K, nbr)
    S = [None] * (K + 1)
    S[K] = set(targets.tolist())
    for k in range(K, 0, -1):
        S[k - 1] = set(S[k])
        for u in S[k]:
            S[k - 1] |= {int(v) for v in nbr[u] if v >= 0}
    for k in range(K + 1):
        assert sets[k].tolist() == sorted(S[k])


def test_layerwise_equals_minibatch(orc):
    # Sec. 3.4: the layer-wise pass computes each node's vector once, and gives
    # the same values as Algorithm 2 run on any target set.
    wl = synth.WORKLOADS["tiny"]
    data = synth.make_workload(wl)
    idx, cnt, wts, _ = orc.build_neighborhoods(data["offsets"], data["col"], wl.num_pins,
                                               wl.seed, wl.walks, wl.hops, wl.T)
    full = orc.embed_all(data["x"], wl.num_pins, data["layers"], idx, wts)
    targets = np.array([0, 5, 1999, 2000, 2499, 1234], np.int32)
    mb = orc.minibatch_embed(targets, data["x"], data["layers"], idx, wts)
    np.testing.assert_allclose(mb, full[targets], rtol=0, atol=1e-14)
    norms = np.linalg.norm(full, axis=1)
    assert np.all(np.abs(norms - 1) < 1e-12)


def test_max_margin_loss_closed_form(orc):
    zq = np.array([[1.0, 0.0]])
    zpos = np.array([[1.0, 0.0]])
    zneg = np.array([[0.0, 1.0], [1.0, 0.0]])
    # neg 1: 0 - 1 + 0.1 < 0 -> 0; neg 2: 1 - 1 + 0.1 = 0.1; mean over 2 negatives.
    loss, per = orc.max_margin_loss(zq, zpos, zneg, 0.1)
    assert loss == pytest.approx(0.05, abs=1e-15)
    # Two pairs; second has its positive orthogonal: each negative costs z_q.z_n + 0.1.
    zq = np.array([[1.0, 0.0], [0.6, 0.8]])
    zpos = np.array([[1.0, 0.0], [0.8, -0.6]])
    zneg = np.array([[0.0, 1.0], [-1.0, 0.0]])
    loss, per = orc.max_margin_loss(zq, zpos, zneg, 0.1)
    want2 = (max(0, 0.8 + 0.1) + max(0, -0.6 + 0.1)) / 2
    np.testing.assert_allclose(per, [0.0, want2], atol=1e-15)
    assert loss == pytest.approx(want2 / 2, abs=1e-15)
    # Well-separated negatives give zero loss.
    loss, _ = orc.max_margin_loss(zq[:1], zpos[:1], np.array([[-1.0, 0.0]]), 0.5)
    assert loss == 0.0


def test_max_margin_loss_with_hard_negatives(orc):
    # Hard negatives join each pair's negative set (Sec. 3.3): a worked example.
    zq = np.array([[1.0, 0.0], [0.6, 0.8]])
    zpos = np.array([[1.0, 0.0], [0.8, -0.6]])
    zneg = np.array([[0.0, 1.0], [-1.0, 0.0]])
    zhard = np.array([[[1.0, 0.0], [0.6, 0.8]], [[0.6, 0.8], [0.0, -1.0]]])
    valid = np.array([[1, 1], [1, 0]], bool)
    loss, per = orc.max_margin_loss(zq, zpos, zneg, 0.1, zhard, valid)
    # Pair 0: shared 0, 0; hard: 1 - 1 + 0.1 = 0.1, 0.6 - 1 + 0.1 < 0 -> 0; mean over 4.
    # Pair 1: shared 0.9, 0; hard 1 + 0.1 = 1.1 (second entry absent); mean over 3.
    np.testing.assert_allclose(per, [0.1 / 4, (0.9 + 1.1) / 3], atol=1e-15)
    assert loss == pytest.approx((0.1 / 4 + 2.0 / 3) / 2, abs=1e-15)
    # No hard entry present: the shared-only loss, exactly.
    l0, p0 = orc.max_margin_loss(zq, zpos, zneg, 0.1)
    l1, p1 = orc.max_margin_loss(zq, zpos, zneg, 0.1, zhard, np.zeros((2, 2), bool))
    assert l1 == l0 and np.array_equal(p1, p0)
    # Hard negatives equal to the shared ones: the mean over the multiset,
    # i.e. the same per-pair terms.
    rng = np.random.default_rng(1)
    zq, zpos, zneg = (rng.standard_normal((3, 8)), rng.standard_normal((3, 8)),
                      rng.standard_normal((5, 8)))
    zh = np.broadcast_to(zneg, (3, 5, 8))
    _, pa = orc.max_margin_loss(zq, zpos, zneg, 0.3)
    _, pb = orc.max_margin_loss(zq, zpos, zneg, 0.3, zh)
    np.testing.assert_allclose(pb, pa, rtol=1e-14)
    # Moving an item from the shared set into every pair's hard set keeps the terms.
    _, pc = orc.max_margin_loss(zq, zpos, zneg[:4], 0.3, np.broadcast_to(zneg[4:], (3, 1, 8)))
    np.testing.assert_allclose(pc, pa, rtol=1e-14)


def test_sampled_route_equals_full_table(orc):
    # The on-demand route (neighbourhoods walked only for the nodes a target set
    # needs, features given only for S^(0)) must reproduce the full-table route.
    wl = synth.WORKLOADS["tiny"]
    data = synth.make_workload(wl)
    idx, cnt, wts, _ = orc.build_neighborhoods(data["offsets"], data["col"], wl.num_pins,
                                               wl.seed, wl.walks, wl.hops, wl.T)
    targets = np.array([3, 2001, 77, 1500, 2499, 3], np.int32)
    smp = orc.minibatch_sample(targets, 2, data["offsets"], data["col"], wl.num_pins, wl.seed,
                               wl.walks, wl.hops, wl.T)
    full_sets = orc.minibatch_sets(targets, 2, idx)
    for a, b in zip(smp["sets"], full_sets):
        np.testing.assert_array_equal(a, b)
    np.testing.assert_array_equal(smp["row_ids"], full_sets[1])
    np.testing.assert_array_equal(smp["idx"], idx[full_sets[1]])
    s0 = smp["sets"][0]
    got = orc.minibatch_embed_sampled(targets, s0, data["x"][s0], smp, data["layers"])
    want = orc.minibatch_embed(targets, data["x"], data["layers"], idx, wts)
    np.testing.assert_array_equal(got, want)
