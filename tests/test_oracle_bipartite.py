"""Pins for the oracle's MapReduce-inference variant (Sec. 3.4): graph
neighbourhoods (boards pool their pins, pins their boards; rows longer than T
sampled) and the all-node embedding with featureless boards.

* Rows of at most T entries equal the CSR rows (ids ascending, weight 1/deg).
* Longer rows: the draws re-derived with the published Philox stream and
  counted with Counter; uniformity of the draws over a long row (chi-square).
* Bipartite structure, weight sums, invalid entries, source subsets.
* Embedding closed form: with Q = I, q = 0, W = [0 | I], w = 0 and
  nonnegative pin features, layer 1 gives each board the normalised mean of
  its pins' features and each pin zero (its boards have no features); layer 2
  gives each pin the normalised mean of its boards' layer-1 vectors --
  written out with numpy from the CSR.
"""

from collections import Counter

import numpy as np

import synth


def _tiny():
    wl = synth.WORKLOADS["tiny"]
    off, col, _ = synth.make_graph(wl)
    return wl, off, col


def test_short_rows_are_csr_rows(orc):
    wl, off, col = _tiny()
    N = wl.num_nodes
    deg = np.diff(off)
    T = 64
    idx, cnt, wts = orc.graph_neighborhoods(off, col, 7, T)
    short = np.nonzero(deg <= T)[0]
    assert len(short) > 2000
    for u in short[::7]:
        row = col[off[u]:off[u + 1]]
        k = len(row)
        np.testing.assert_array_equal(idx[u, :k], np.sort(row))
        assert np.all(idx[u, k:] == -1) and np.all(cnt[u, :k] == 1) and np.all(cnt[u, k:] == 0)
        np.testing.assert_array_equal(wts[u, :k], np.full(k, np.float32(1) / np.float32(k)))
    # Bipartite: pins list boards, boards list pins.
    pins_rows = idx[: wl.num_pins]
    assert np.all((pins_rows == -1) | (pins_rows >= wl.num_pins))
    boards_rows = idx[wl.num_pins:]
    assert np.all((boards_rows == -1) | ((boards_rows >= 0) & (boards_rows < wl.num_pins)))
    s = wts.astype(np.float64).sum(axis=1)
    live = cnt[:, 0] > 0
    assert np.all(np.abs(s[live] - 1) <= T * 2.0**-24) and np.all(s[~live] == 0)
    assert live.sum() == np.count_nonzero(deg)
    assert N == len(idx)


def test_long_rows_brute_force(orc):
    wl, off, col = _tiny()
    deg = np.diff(off)
    seed, T = 99, 8
    idx, cnt, wts = orc.graph_neighborhoods(off, col, seed, T)
    key = [seed & 0xFFFFFFFF, seed >> 32]
    long_rows = np.nonzero(deg > T)[0]
    assert len(long_rows) > 100
    for u in long_rows[::5]:
        row = col[off[u]:off[u + 1]]
        picks = [int(row[(int(orc.philox4x32_10([int(u), j, 0, 2], key)[0]) * len(row)) >> 32])
                 for j in range(T)]
        c = sorted(Counter(picks).items())
        k = len(c)
        np.testing.assert_array_equal(idx[u, :k], [v for v, _ in c])
        np.testing.assert_array_equal(cnt[u, :k], [n for _, n in c])
        np.testing.assert_array_equal(wts[u, :k], [np.float32(n) / np.float32(T) for _, n in c])
        assert np.all(idx[u, k:] == -1)


def test_sampling_is_uniform_over_a_long_row(orc):
    P, B = 1000, 1
    off, col = synth.csr_from_edges(P, B, [(p, 0) for p in range(P)])
    T = 250
    counts = np.zeros(P)
    for seed in range(40):
        idx, cnt, _ = orc.graph_neighborhoods(off, col, seed, T, sources=np.array([P], np.int32))
        k = cnt[0] > 0
        counts[idx[0, k]] += cnt[0, k]
    assert counts.sum() == 40 * T
    e = counts.sum() / P
    chi2 = float(((counts - e) ** 2 / e).sum())
    assert chi2 < (P - 1) + 6 * np.sqrt(2 * (P - 1)), chi2


def test_subsets_invalid_sources_and_entries(orc):
    wl, off, col = _tiny()
    full = orc.graph_neighborhoods(off, col, 3, 10)
    src = np.array([2400, 5, -1, 2500, 17, 2400], np.int32)
    sub = orc.graph_neighborhoods(off, col, 3, 10, sources=src)
    for r, u in enumerate(src):
        if 0 <= u < wl.num_nodes:
            for a, b in zip(sub, full):
                np.testing.assert_array_equal(a[r], b[u])
        else:
            assert np.all(sub[0][r] == -1) and np.all(sub[1][r] == 0) and np.all(sub[2][r] == 0)
    # An entry outside the graph is dropped and the rest renormalised.
    off2 = np.array([0, 3, 4, 5, 6], np.int64)
    col2 = np.array([2, 99, 3, 0, 0, 0], np.int32)
    idx, cnt, wts = orc.graph_neighborhoods(off2, col2, 1, 4)
    np.testing.assert_array_equal(idx[0, :2], [2, 3])
    np.testing.assert_array_equal(wts[0, :2], [0.5, 0.5])


def test_embedding_closed_form(orc):
    wl, off, col = _tiny()
    P, N, d = wl.num_pins, wl.num_nodes, 16
    rng = np.random.default_rng(2)
    x = np.abs(rng.standard_normal((P, d)))
    deg = np.diff(off)
    T = int(deg.max())
    idx, cnt, wts = orc.graph_neighborhoods(off, col, 0, T)
    eye = np.eye(d)
    L = {"Q": eye, "q": np.zeros(d), "W": np.hstack([np.zeros((d, d)), eye]), "w": np.zeros(d)}
    h = orc.embed_all_bipartite(x, N, [L, L], idx, wts)

    def normalize(a):
        n = np.linalg.norm(a, axis=1, keepdims=True)
        return np.where(n > 0, a / np.where(n > 0, n, 1), 0.0)

    h1 = np.zeros((N, d))
    for b in range(P, N):
        nb = col[off[b]:off[b + 1]]
        if len(nb):
            h1[b] = x[nb].mean(axis=0)
    h1 = normalize(h1)  # pins: zero (their boards have no features)
    want = np.zeros((N, d))
    for p in range(P):
        nb = col[off[p]:off[p + 1]]
        if len(nb):
            want[p] = h1[nb].mean(axis=0)
    want = normalize(want)  # boards: zero (their pins are zero at layer 1)
    np.testing.assert_allclose(h, want, rtol=0, atol=1e-12)
    assert np.abs(np.linalg.norm(h[:P], axis=1) - 1).max() < 1e-12
