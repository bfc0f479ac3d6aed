"""Pins for the oracle's hard negative items (Sec. 3.3).

* Brute force: the PPR ranking (visit counts of the query's walks, count
  descending, ties to the lower id) re-derived with Counter and sorted from the
  raw visit list; every drawn item sits in the rank window, at the position the
  published Philox stream selects.
* PPR reading: with many walks the visit-count ranking agrees with the
  closed-form expected visit counts wherever those are far apart.
* Uniformity: many draws over one window pass a chi-square bound.
* Special cases: the window [0, T) stays inside the top-T neighbourhood;
  empty windows, isolated and out-of-range queries give -1; rows depend only on
  their own query.
"""

from collections import Counter

import numpy as np

import synth

from test_oracle_walks import EDGES_SMALL, _expected_counts, _transition


def _ranked(visits):
    cnt = Counter(visits.tolist())
    return [v for v, _ in sorted(cnt.items(), key=lambda kv: (-kv[1], kv[0]))]


def _tiny():
    wl = synth.WORKLOADS["tiny"]
    off, col, _ = synth.make_graph(wl)
    return wl, off, col


def test_hard_negatives_brute_force(orc):
    wl, off, col = _tiny()
    P = wl.num_pins
    seed, walks, hops, lo, hi, k = 77, 300, 3, 20, 60, 9
    rng = np.random.default_rng(4)
    q = np.concatenate([rng.choice(P, 25, replace=False),
                        P + rng.choice(wl.num_boards, 10, replace=False)]).astype(np.int32)
    got = orc.hard_negatives(off, col, P, seed, walks, hops, q, lo, hi, k)
    assert got.shape == (len(q), k)
    key = [seed & 0xFFFFFFFF, seed >> 32]
    for i, u in enumerate(q):
        visits, _ = orc.walk_visits(off, col, P, seed, int(u), walks, hops)
        order = _ranked(visits)
        window = order[lo:min(hi, len(order))]
        assert len(window) > 0
        for j in range(k):
            r0 = int(orc.philox4x32_10([int(u), j, 0, 1], key)[0])
            assert got[i, j] == window[(r0 * len(window)) >> 32], (u, j)
        assert set(got[i].tolist()) <= set(window)
        assert int(u) not in got[i]
        assert np.all(got[i] < P)


def test_visit_ranking_follows_expected_counts(orc):
    P, B = 8, 5
    off, col = synth.csr_from_edges(P, B, EDGES_SMALL)
    A = _transition(off, col)
    walks, hops = 40000, 3
    for u in range(P):
        exp = _expected_counts(A, u, P, walks, hops)
        visits, _ = orc.walk_visits(off, col, P, 23, u, walks, hops)
        order = _ranked(visits)
        rank = {v: r for r, v in enumerate(order)}
        sig = np.sqrt(hops * np.maximum(exp, 1.0))
        for a in range(P):
            for b in range(P):
                if exp[a] > exp[b] + 10 * (sig[a] + sig[b]) and exp[b] > 0:
                    assert rank[a] < rank[b], (u, a, b)
    # Window of ranks 1-3 from pin 3: the draws land only on those ranks.
    visits, _ = orc.walk_visits(off, col, P, 23, 3, walks, hops)
    order = _ranked(visits)
    got = orc.hard_negatives(off, col, P, 23, walks, hops, np.array([3], np.int32), 1, 4, 64)
    assert set(got[0].tolist()) == set(order[1:4])


def test_hard_negative_draws_are_uniform(orc):
    wl, off, col = _tiny()
    P = wl.num_pins
    lo, hi, k = 10, 50, 40000
    q = np.array([17], np.int32)
    got = orc.hard_negatives(off, col, P, 5, 400, 3, q, lo, hi, k)
    visits, _ = orc.walk_visits(off, col, P, 5, 17, 400, 3)
    window = _ranked(visits)[lo:hi]
    n = len(window)
    assert n == hi - lo
    pos = {v: i for i, v in enumerate(window)}
    c = np.bincount([pos[v] for v in got[0].tolist()], minlength=n).astype(float)
    e = k / n
    chi2 = float(((c - e) ** 2 / e).sum())
    assert chi2 < (n - 1) + 6 * np.sqrt(2 * (n - 1)), chi2


def test_window_top_t_inside_neighbourhood(orc):
    wl, off, col = _tiny()
    P = wl.num_pins
    seed, walks, hops, T = 9, 200, 2, 10
    idx, cnt, _, _ = orc.build_neighborhoods(off, col, P, seed, walks, hops, T)
    q = np.arange(0, P + wl.num_boards, 37, dtype=np.int32)
    got = orc.hard_negatives(off, col, P, seed, walks, hops, q, 0, T, 16)
    for i, u in enumerate(q):
        top = set(idx[u][idx[u] >= 0].tolist())
        assert set(got[i].tolist()) <= top, u


def test_degenerate_queries_and_windows(orc):
    P, B = 3, 2
    off, col = synth.csr_from_edges(P, B, [(0, 0), (1, 0)])  # pin 2, board 1 isolated
    q = np.array([0, 2, 4, -1, 5, 1, 0], np.int32)
    got = orc.hard_negatives(off, col, P, 1, 10, 2, q, 0, 5, 3)
    assert np.all(got[0] == 1) and np.all(got[5] == 0) and np.all(got[6] == 1)
    assert np.all(got[[1, 2, 3, 4]] == -1)
    # A window past the ranked pins is empty.
    assert np.all(orc.hard_negatives(off, col, P, 1, 10, 2, q, 1, 5, 3) == -1)
    assert orc.hard_negatives(off, col, P, 1, 10, 2, q, 0, 5, 0).shape == (len(q), 0)


def test_rows_depend_on_their_query_only(orc):
    wl, off, col = _tiny()
    P = wl.num_pins
    q = np.array([5, 900, 1999, 2100, 5, 42], np.int32)
    full = orc.hard_negatives(off, col, P, 3, 300, 3, q, 30, 90, 7)
    for i, u in enumerate(q):
        one = orc.hard_negatives(off, col, P, 3, 300, 3, np.array([u], np.int32), 30, 90, 7)
        np.testing.assert_array_equal(one[0], full[i])
    np.testing.assert_array_equal(full[0], full[4])
    # A wider window starting at the same rank keeps draws in the larger range.
    wide = orc.hard_negatives(off, col, P, 3, 300, 3, q, 30, 200, 7)
    assert not np.array_equal(wide, full)
