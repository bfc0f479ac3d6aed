"""Seeded generators for bipartite pin-board graphs, features and parameters.

Node ids: pins are [0, P), boards are [P, P + B). The graph is stored as an
undirected CSR with both directions: a pin row lists its boards, a board row
lists its pins, every row sorted ascending, no duplicate edges.

Degree model (matching the five workloads this library is exercised on):
  * pin degree: Uniform{1..8} (tiny graph) or Zipf(a) clipped to [1, hi];
  * board choice per edge: uniform, or rank-Zipf(b) -- board of popularity
    rank r is drawn with probability proportional to r^-b, ranks mapped to ids
    by a seeded permutation; a pin's boards are distinct (duplicates redrawn).
Features: pins N(0,1); a board's feature is the mean of its pins' features
(zero for a board without pins). Layer parameters: Glorot-uniform matrices,
biases U(-0.1, 0.1).
"""

from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Optional

import numpy as np
import torch


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    num_pins: int
    num_boards: int
    pin_degree: str           # "uniform8" or "zipf"
    zipf_a: float             # pin-degree exponent (zipf)
    degree_hi: int            # pin-degree clip
    board_zipf: Optional[float]  # None = uniform boards
    d_in: int
    m: int
    d_out: int
    K: int
    walks: int
    hops: int
    T: int
    dtype: str                # "f32" or "bf16"
    seed: int
    offsets64: bool = False

    @property
    def num_nodes(self) -> int:
        return self.num_pins + self.num_boards

    def scaled(self, num_pins: int, num_boards: int, name: Optional[str] = None) -> "Workload":
        return dataclasses.replace(self, num_pins=num_pins, num_boards=num_boards,
                                   name=name or f"{self.name}-scaled")


# The five workloads: a tiny graph, a 1.2M-node graph in fp32, a 12M-node graph
# with wide bf16 features, the minibatch-shaped forward on the 1.2M-node graph,
# and the largest single-GPU shard (100M nodes, int64 row offsets).
WORKLOADS: Dict[str, Workload] = {
    "tiny": Workload("tiny", 2000, 500, "uniform8", 0.0, 8, None, 64, 64, 64, 2, 200, 2, 10,
                     "f32", 1),
    "medium": Workload("medium", 1_000_000, 200_000, "zipf", 2.0, 500, 1.5, 256, 512, 256, 2,
                       100, 3, 50, "f32", 2),
    "large": Workload("large", 10_000_000, 2_000_000, "zipf", 2.0, 2000, 1.5, 1024, 2048, 512,
                      2, 100, 3, 50, "bf16", 3),
    # Same graph and walk seed as "medium" (the minibatch forward runs on that
    # graph), bf16 storage.
    "minibatch": Workload("minibatch", 1_000_000, 200_000, "zipf", 2.0, 500, 1.5, 256, 512,
                          256, 2, 100, 3, 50, "bf16", 2),
    "shard": Workload("shard", 80_000_000, 20_000_000, "zipf", 2.0, 5000, 1.5, 256, 512, 256,
                      2, 50, 3, 50, "bf16", 5, offsets64=True),
}


def bf16_round(a: np.ndarray) -> np.ndarray:
    """Round fp32 values to the nearest bfloat16 (ties to even); returned as fp32."""
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    return t.to(torch.bfloat16).to(torch.float32).numpy()


def _pin_degrees(wl: Workload, rng: np.random.Generator) -> np.ndarray:
    if wl.pin_degree == "uniform8":
        return rng.integers(1, 9, size=wl.num_pins, dtype=np.int64)
    deg = rng.zipf(wl.zipf_a, size=wl.num_pins)
    return np.clip(deg, 1, wl.degree_hi).astype(np.int64)


def _draw_boards(wl: Workload, rng: np.random.Generator, n: int, cdf: Optional[np.ndarray],
                 perm: Optional[np.ndarray]) -> np.ndarray:
    if cdf is None:
        return rng.integers(0, wl.num_boards, size=n, dtype=np.int64)
    u = rng.random(n)
    rank = np.searchsorted(cdf, u, side="right")
    rank = np.minimum(rank, wl.num_boards - 1)
    return perm[rank]


def make_graph(wl: Workload):
    """Returns (offsets int64 [N+1], col int32 [nnz], num_edges). Deterministic in wl.seed."""
    rng = np.random.default_rng([wl.seed, 1])
    P, B = wl.num_pins, wl.num_boards
    deg = _pin_degrees(wl, rng)
    deg = np.minimum(deg, B)
    cdf = perm = None
    if wl.board_zipf is not None:
        r = np.arange(1, B + 1, dtype=np.float64)
        p = r ** (-wl.board_zipf)
        cdf = np.cumsum(p)
        cdf /= cdf[-1]
        perm = rng.permutation(B).astype(np.int64)
    E = int(deg.sum())
    pin = np.repeat(np.arange(P, dtype=np.int64), deg)
    board = _draw_boards(wl, rng, E, cdf, perm)
    # Redraw duplicate (pin, board) pairs until every pin's boards are distinct:
    # a few vectorised passes over the pins that still hold a duplicate, then a
    # per-pin pass (first-drawn order kept) for the few heavy pins left.
    sel = np.arange(E, dtype=np.int64)
    for _ in range(8):
        key = pin[sel] * B + board[sel]
        order = np.argsort(key, kind="stable")
        ks = key[order]
        dup_sorted = np.zeros(len(sel), bool)
        dup_sorted[1:] = ks[1:] == ks[:-1]
        if not dup_sorted.any():
            sel = sel[:0]
            break
        dup = sel[order[dup_sorted]]
        board[dup] = _draw_boards(wl, rng, len(dup), cdf, perm)
        sel = sel[np.isin(pin[sel], np.unique(pin[dup]))]
    if len(sel):
        starts = np.concatenate([[0], np.cumsum(deg)])
        for p in np.unique(pin[sel]):
            lo, hi = int(starts[p]), int(starts[p + 1])
            chosen = list(dict.fromkeys(board[lo:hi].tolist()))
            seen = set(chosen)
            while len(chosen) < hi - lo:
                for b in _draw_boards(wl, rng, 2 * (hi - lo - len(chosen)) + 8, cdf, perm).tolist():
                    if b not in seen and len(chosen) < hi - lo:
                        seen.add(b)
                        chosen.append(b)
            board[lo:hi] = chosen
    key = pin * B + board
    order = np.argsort(key, kind="stable")
    pin, board = pin[order], board[order]
    # Pin rows (boards ascending) then board rows (pins ascending).
    bo = np.lexsort((pin, board))
    board_pins = pin[bo]
    board_deg = np.bincount(board, minlength=B).astype(np.int64)
    offsets = np.zeros(P + B + 1, np.int64)
    offsets[1:P + 1] = np.cumsum(deg)
    offsets[P + 1:] = offsets[P] + np.cumsum(board_deg)
    col = np.empty(2 * E, np.int32)
    col[:E] = (board + P).astype(np.int32)
    col[E:] = board_pins.astype(np.int32)
    return offsets, col, E


def make_features(wl: Workload, offsets: np.ndarray, col: np.ndarray) -> np.ndarray:
    """Node features [N, d_in] fp32 (already rounded to bf16 when wl.dtype is bf16)."""
    rng = np.random.default_rng([wl.seed, 2])
    P, B, d = wl.num_pins, wl.num_boards, wl.d_in
    x = np.empty((P + B, d), np.float32)
    x[:P] = rng.standard_normal((P, d), dtype=np.float32)
    if wl.dtype == "bf16":
        x[:P] = bf16_round(x[:P])
    # Board features: mean of the board's pins, accumulated in fp64.
    import scipy.sparse as sp
    b_off = offsets[P:] - offsets[P]
    b_col = col[offsets[P]:]
    if len(b_col):
        A = sp.csr_matrix((np.ones(len(b_col)), b_col.astype(np.int64), b_off), shape=(B, P))
        sums = np.asarray(A @ x[:P].astype(np.float64))
        cnt = np.diff(b_off).astype(np.float64)
        mean = np.where(cnt[:, None] > 0, sums / np.maximum(cnt, 1)[:, None], 0.0)
    else:
        mean = np.zeros((B, d))
    x[P:] = mean.astype(np.float32)
    if wl.dtype == "bf16":
        x[P:] = bf16_round(x[P:])
    return x


def make_layers(wl: Workload, seed_offset: int = 0) -> List[dict]:
    """K layers of (Q [m, d_in], q [m], W [d_out, d_in + m], w [d_out]) as fp32 numpy;
    Q and W are rounded to bf16 when wl.dtype is bf16 (biases stay fp32)."""
    rng = np.random.default_rng([wl.seed, 3, seed_offset])
    layers = []
    d_prev = wl.d_in
    for _ in range(wl.K):
        m, d = wl.m, wl.d_out
        aq = math.sqrt(6.0 / (d_prev + m))
        aw = math.sqrt(6.0 / (d_prev + m + d))
        Q = rng.uniform(-aq, aq, size=(m, d_prev)).astype(np.float32)
        q = rng.uniform(-0.1, 0.1, size=m).astype(np.float32)
        W = rng.uniform(-aw, aw, size=(d, d_prev + m)).astype(np.float32)
        w = rng.uniform(-0.1, 0.1, size=d).astype(np.float32)
        if wl.dtype == "bf16":
            Q, W = bf16_round(Q), bf16_round(W)
        layers.append({"Q": Q, "q": q, "W": W, "w": w})
        d_prev = d
    return layers


def make_mlp(d_in: int, d_hidden: int, d_out: int, seed: int, dtype: str = "f32") -> dict:
    """Output dense layers (G1 [d_hidden, d_in], g [d_hidden], G2 [d_out, d_hidden])
    as fp32 numpy: Glorot-uniform matrices, g ~ U(-0.1, 0.1); G1 and G2 rounded to
    bf16 for bf16 storage."""
    rng = np.random.default_rng([seed, 5])
    a1 = math.sqrt(6.0 / (d_in + d_hidden))
    a2 = math.sqrt(6.0 / (d_hidden + d_out))
    G1 = rng.uniform(-a1, a1, size=(d_hidden, d_in)).astype(np.float32)
    g = rng.uniform(-0.1, 0.1, size=d_hidden).astype(np.float32)
    G2 = rng.uniform(-a2, a2, size=(d_out, d_hidden)).astype(np.float32)
    if dtype == "bf16":
        G1, G2 = bf16_round(G1), bf16_round(G2)
    return {"G1": G1, "g": g, "G2": G2}


def make_workload(wl: Workload):
    """Full input bundle: dict with offsets, col, num_edges, x, layers."""
    offsets, col, E = make_graph(wl)
    x = make_features(wl, offsets, col)
    return {"wl": wl, "offsets": offsets, "col": col, "num_edges": E, "x": x,
            "layers": make_layers(wl)}


def minibatch_pairs(wl: Workload, offsets: np.ndarray, col: np.ndarray, batch: int,
                    num_neg: int, seed: int = 0):
    """Training pairs for one minibatch: `batch` query pins drawn uniformly
    without replacement, each paired with a positive pin that shares one of its
    boards (a board drawn uniformly among the query's boards, then a pin other
    than the query drawn uniformly from that board) -- a stand-in for the
    engagement pairs the paper trains on -- and `num_neg` shared negative pins
    drawn uniformly. Queries whose boards hold no other pin are redrawn."""
    rng = np.random.default_rng([wl.seed, 4, seed])
    P = wl.num_pins
    queries, positives = [], []
    taken = set()
    while len(queries) < batch:
        for q in rng.choice(P, size=2 * (batch - len(queries)) + 8, replace=False).tolist():
            if q in taken or len(queries) == batch:
                continue
            lo, hi = int(offsets[q]), int(offsets[q + 1])
            if hi == lo:
                continue
            b = int(col[lo + rng.integers(0, hi - lo)])
            blo, bhi = int(offsets[b]), int(offsets[b + 1])
            if bhi - blo < 2:
                continue
            while True:
                v = int(col[blo + rng.integers(0, bhi - blo)])
                if v != q:
                    break
            taken.add(q)
            queries.append(q)
            positives.append(v)
    negatives = rng.integers(0, P, size=num_neg)
    return (np.asarray(queries, np.int32), np.asarray(positives, np.int32),
            negatives.astype(np.int32))


def csr_from_edges(num_pins: int, num_boards: int, edges) -> tuple:
    """Undirected CSR (offsets int64, col int32) from (pin, board_index) pairs,
    board_index in [0, num_boards); rows sorted, duplicates dropped."""
    e = np.unique(np.asarray(edges, dtype=np.int64).reshape(-1, 2), axis=0)
    N = num_pins + num_boards
    src = np.concatenate([e[:, 0], e[:, 1] + num_pins])
    dst = np.concatenate([e[:, 1] + num_pins, e[:, 0]])
    order = np.lexsort((dst, src))
    src, dst = src[order], dst[order]
    offsets = np.zeros(N + 1, np.int64)
    offsets[1:] = np.cumsum(np.bincount(src, minlength=N))
    return offsets, dst.astype(np.int32)


def random_neighborhoods(n_rows: int, n_transform: int, T: int, seed: int,
                         fill: float = 0.9):
    """An arbitrary neighbourhood table as layer input: per row k <= T distinct
    ids in [0, n_transform) (k = 0 for about (1 - fill) of the rows), padding
    -1 at the tail, counts in 1..9 and independent positive weights in
    [0.05, 1) (not normalised: a layer takes any weights)."""
    rng = np.random.default_rng([seed, 5])
    idx = np.full((n_rows, T), -1, np.int32)
    counts = np.zeros((n_rows, T), np.uint16)
    weights = np.zeros((n_rows, T), np.float32)
    live = rng.random(n_rows) < fill
    ks = np.where(live, rng.integers(1, min(T, n_transform) + 1, size=n_rows), 0)
    for r in np.nonzero(ks)[0]:
        k = int(ks[r])
        idx[r, :k] = rng.choice(n_transform, size=k, replace=False)
        counts[r, :k] = np.sort(rng.integers(1, 10, size=k))[::-1]
        weights[r, :k] = rng.uniform(0.05, 1.0, size=k).astype(np.float32)
    return idx, counts, weights
