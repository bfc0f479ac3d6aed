"""Pins for the oracle's importance neighbourhoods (Sec. 3.2).

* Closed form: on small bipartite graphs the expected visit count of pin v in
  W walks from u is W * sum_h (A^{s_h})[u, v], A the row-stochastic transition
  matrix and s_h the edge step of the h-th pin landing (2h from a pin, 2h-1
  from a board). Counts must fall within 5 sigma of it.
* Star board (special case): every other pin is equally likely.
* Brute force: top-T, tie order and weights re-derived from the raw visit list
  with Python's Counter and sorted.
* Exact step totals, self exclusion, weight sums, source-subset consistency.
"""

from collections import Counter

import numpy as np
import pytest

import synth

EDGES_SMALL = [(0, 0), (0, 1), (1, 0), (2, 0), (2, 2), (3, 1), (3, 2), (3, 3), (4, 3), (5, 2),
               (6, 1), (7, 3), (7, 0)]


def _transition(offsets, col):
    N = len(offsets) - 1
    A = np.zeros((N, N))
    for i in range(N):
        lo, hi = offsets[i], offsets[i + 1]
        for j in col[lo:hi]:
            A[i, j] += 1.0 / (hi - lo)
    return A


def _expected_counts(A, u, num_pins, walks, hops):
    N = A.shape[0]
    e = np.zeros(N)
    e[u] = 1.0
    exp = np.zeros(N)
    land_steps = [2 * h for h in range(1, hops + 1)] if u < num_pins else \
        [2 * h - 1 for h in range(1, hops + 1)]
    dist = e.copy()
    for s in range(1, max(land_steps) + 1):
        dist = dist @ A
        if s in land_steps:
            exp += walks * dist
    exp[num_pins:] = 0.0
    exp[u] = 0.0
    return exp


@pytest.mark.parametrize("graph", ["small", "star"])
def test_visit_counts_match_closed_form(orc, graph):
    if graph == "small":
        P, B = 8, 5  # board 4 has no pins
        off, col = synth.csr_from_edges(P, B, EDGES_SMALL)
    else:
        P, B = 12, 1
        off, col = synth.csr_from_edges(P, B, [(p, 0) for p in range(P)])
    A = _transition(off, col)
    walks, hops = 40000, 3
    for u in range(P + B):
        visits, steps = orc.walk_visits(off, col, P, seed=11, u=u, walks=walks, hops=hops)
        got = np.bincount(visits, minlength=P + B).astype(float)
        exp = _expected_counts(A, u, P, walks, hops)
        tol = 5.0 * np.sqrt(hops * exp) + 1.0
        assert np.all(np.abs(got - exp) <= tol), (u, got, exp)
        assert got[u] == 0  # the source is never its own neighbour
        assert np.all(got[P:] == 0)  # only pins are recorded
        deg = off[u + 1] - off[u]
        want_steps = 0 if deg == 0 else walks * (2 * hops if u < P else 2 * hops - 1)
        assert steps == want_steps
    if graph == "star":
        # Special case: from any pin all other pins are equally likely.
        visits, _ = orc.walk_visits(off, col, P, seed=3, u=0, walks=walks, hops=hops)
        c = np.bincount(visits, minlength=P)[1:P]
        mean = walks * hops / P
        assert np.all(np.abs(c - mean) <= 5 * np.sqrt(hops * mean) + 1)


def _brute_top_t(visits, T):
    cnt = Counter(visits.tolist())
    order = sorted(cnt.items(), key=lambda kv: (-kv[1], kv[0]))[:T]
    S = sum(c for _, c in order)
    idx = [v for v, _ in order] + [-1] * (T - len(order))
    counts = [c for _, c in order] + [0] * (T - len(order))
    w = [np.float32(c) / np.float32(S) for _, c in order] + [np.float32(0)] * (T - len(order))
    return np.array(idx, np.int32), np.array(counts, np.uint16), np.array(w, np.float32)


def test_top_t_matches_brute_force(orc):
    wl = synth.WORKLOADS["tiny"]
    off, col, _ = synth.make_graph(wl)
    P = wl.num_pins
    idx, cnt, wts, steps = orc.build_neighborhoods(off, col, P, wl.seed, wl.walks, wl.hops, wl.T)
    rng = np.random.default_rng(0)
    rows = np.concatenate([rng.choice(P, 60, replace=False),
                           P + rng.choice(wl.num_boards, 40, replace=False)])
    for u in rows:
        visits, _ = orc.walk_visits(off, col, P, wl.seed, int(u), wl.walks, wl.hops)
        bi, bc, bw = _brute_top_t(visits, wl.T)
        np.testing.assert_array_equal(idx[u], bi)
        np.testing.assert_array_equal(cnt[u], bc)
        np.testing.assert_array_equal(wts[u].view(np.uint32), bw.view(np.uint32))
    # Every pin has at least one board in this graph, so every walk runs to the end.
    deg = np.diff(off)
    n_board_live = int(np.count_nonzero(deg[P:]))
    assert steps == wl.walks * (P * 2 * wl.hops + n_board_live * (2 * wl.hops - 1))


def test_weights_rows_and_subsets(orc):
    wl = synth.WORKLOADS["tiny"]
    off, col, _ = synth.make_graph(wl)
    P = wl.num_pins
    idx, cnt, wts, _ = orc.build_neighborhoods(off, col, P, 5, 30, 2, 16)
    live = cnt[:, 0] > 0
    s = wts.astype(np.float64).sum(axis=1)
    assert np.all(np.abs(s[live] - 1.0) <= 16 * 2.0**-24)
    assert np.all(s[~live] == 0)
    # Ranks are ordered by (count desc, id asc); padding only at the tail.
    for r in range(len(idx)):
        k = int(np.count_nonzero(idx[r] >= 0))
        assert np.all(idx[r, k:] == -1) and np.all(cnt[r, k:] == 0)
        pairs = list(zip((-cnt[r, :k].astype(int)).tolist(), idx[r, :k].tolist()))
        assert pairs == sorted(pairs)
        assert r not in idx[r, :k]
        assert np.all(idx[r, :k] < P)
    src = np.array([2400, 3, 1999, 7, 7, 2000], np.int32)
    i2, c2, w2, _ = orc.build_neighborhoods(off, col, P, 5, 30, 2, 16, sources=src)
    np.testing.assert_array_equal(i2, idx[src])
    np.testing.assert_array_equal(c2, cnt[src])
    np.testing.assert_array_equal(w2.view(np.uint32), wts[src].view(np.uint32))


def test_dead_end_and_degenerate_sources(orc):
    P, B = 3, 2
    off, col = synth.csr_from_edges(P, B, [(0, 0), (1, 0)])  # pin 2 and board 1 isolated
    idx, cnt, wts, steps = orc.build_neighborhoods(off, col, P, 1, 10, 2, 4)
    assert np.all(idx[2] == -1) and np.all(idx[4] == -1)
    assert np.all(wts[2] == 0) and np.all(cnt[4] == 0)
    # From pin 0 the only other reachable pin is pin 1.
    assert idx[0, 0] == 1 and np.all(idx[0, 1:] == -1) and wts[0, 0] == 1.0
    # pins 0, 1: 10 walks x 4 steps; board 0: 10 walks x 3 steps; isolated: 0.
    assert steps == 10 * 4 * 2 + 10 * 3
