"""PinSage CPU oracle — TEST INFRASTRUCTURE ONLY.

A plain, slow CPU statement of the PinSage hot path (Ying et al., KDD 2018),
written from the paper: random-walk importance neighbourhoods (Sec. 3.2),
CONVOLVE (Algorithm 1), stacked layers evaluated layer-wise (Secs. 3.2, 3.4),
MINIBATCH (Algorithm 2) with its output dense layers, the aggregators gamma
(importance pooling, and the mean and max of Sec. 4's variants), the hard
negative items of Sec. 3.3 and the max-margin loss (Sec. 3.3, Eq. 1). The
arithmetic lives in ``oracle.cpp`` (fp64; importance weights fp32); this module
only loads that library and marshals numpy arrays.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package. It shares no code with the GPU library in
``paper_1806_01973_amd``; the only thing both sides consume is the seeded input
generator in ``synth``.
"""

from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.cpp")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None


def build(verbose: bool = False) -> str:
    """Compile oracle.cpp with g++ (-O2, IEEE arithmetic, no fast-math)."""
    cmd = ["g++", "-O2", "-std=c++17", "-fPIC", "-shared", "-pthread",
           "-fno-fast-math", "-ffp-contract=off", _SRC, "-o", _LIB_PATH + ".tmp"]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(_LIB_PATH + ".tmp", _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC):
        build()
    lib = ctypes.CDLL(_LIB_PATH)
    P = ctypes.c_void_p
    i64, i32, u64, u32 = ctypes.c_int64, ctypes.c_int, ctypes.c_uint64, ctypes.c_uint32
    lib.orc_philox4x32_10.argtypes = [P, P, P]
    lib.orc_philox4x32_10.restype = None
    lib.orc_walk_word.argtypes = [u64, u32, u32, u32]
    lib.orc_walk_word.restype = u32
    lib.orc_walk_visits.argtypes = [P, P, i64, i64, u64, i64, i32, i32, P, P]
    lib.orc_walk_visits.restype = i64
    lib.orc_build_neighborhoods.argtypes = [P, P, i64, i64, u64, i32, i32, i32, P, i64,
                                            P, P, P, P, i32]
    lib.orc_build_neighborhoods.restype = None
    lib.orc_convolve_layer.argtypes = [P, i64, i32, i64, P, P, i32, P, P, i32, P, P, i32,
                                       P, i64, P, i32, i32]
    lib.orc_convolve_layer.restype = None
    lib.orc_minibatch_sets.argtypes = [P, i64, i32, P, i32, P, P, i64]
    lib.orc_minibatch_sets.restype = i64
    lib.orc_minibatch_embed.argtypes = [P, i64, i32, P, i32, P, P, i32, P, P, P, P, P, P, P,
                                        i32, P]
    lib.orc_minibatch_embed.restype = None
    lib.orc_minibatch_sample.argtypes = [P, i64, i32, P, P, i64, i64, u64, i32, i32, i32, i32]
    lib.orc_minibatch_sample.restype = ctypes.c_void_p
    lib.orc_sample_sizes.argtypes = [P, i32, P]
    lib.orc_sample_sizes.restype = None
    lib.orc_sample_copy.argtypes = [P, i32, P, P, P, P]
    lib.orc_sample_copy.restype = None
    lib.orc_sample_free.argtypes = [P]
    lib.orc_sample_free.restype = None
    lib.orc_minibatch_embed_sampled.argtypes = [P, i64, i32, P, i64, P, i32, P, i64, P, P, i32,
                                                P, P, P, P, P, P, P, i32, P]
    lib.orc_minibatch_embed_sampled.restype = None
    lib.orc_graph_neighborhoods.argtypes = [P, P, i64, u64, i32, P, i64, P, P, P, i32]
    lib.orc_graph_neighborhoods.restype = None
    lib.orc_hard_negatives.argtypes = [P, P, i64, i64, u64, i32, i32, P, i64, i32, i32, i32, P,
                                       i32]
    lib.orc_hard_negatives.restype = None
    lib.orc_output_mlp.argtypes = [P, i64, i32, P, P, i32, P, i32, P, i32]
    lib.orc_output_mlp.restype = None
    lib.orc_max_margin_loss.argtypes = [P, P, i64, P, i64, i32, ctypes.c_double, P]
    lib.orc_max_margin_loss.restype = ctypes.c_double
    lib.orc_max_margin_loss_hard.argtypes = [P, P, i64, P, i64, P, P, i64, i32, ctypes.c_double,
                                             P]
    lib.orc_max_margin_loss_hard.restype = ctypes.c_double
    _lib = lib
    return lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def default_threads() -> int:
    return max(1, len(os.sched_getaffinity(0)))


def philox4x32_10(ctr, key) -> np.ndarray:
    """Philox4x32-10 block function (Salmon et al., SC'11)."""
    lib = _load()
    c = _c(ctr, np.uint32)
    k = _c(key, np.uint32)
    out = np.zeros(4, np.uint32)
    lib.orc_philox4x32_10(_ptr(c), _ptr(k), _ptr(out))
    return out


def walk_word(seed: int, u: int, w: int, s: int) -> int:
    return int(_load().orc_walk_word(seed, u, w, s))


def walk_visits(offsets, col, num_pins, seed, u, walks, hops):
    """Raw pin visits of all walks from u (source excluded) and the edge steps taken."""
    lib = _load()
    off = _c(offsets, np.int64)
    cl = _c(col, np.int32)
    buf = np.zeros(max(1, walks * hops), np.int32)
    steps = np.zeros(1, np.int64)
    n = lib.orc_walk_visits(_ptr(off), _ptr(cl), num_pins, len(off) - 1, seed, u, walks, hops,
                            _ptr(buf), _ptr(steps))
    return buf[:n].copy(), int(steps[0])


def build_neighborhoods(offsets, col, num_pins, seed, walks, hops, T, sources=None,
                        nthreads=None):
    """Importance neighbourhoods (Sec. 3.2): (idx int32, counts uint16, weights fp32, steps)."""
    lib = _load()
    off = _c(offsets, np.int64)
    cl = _c(col, np.int32)
    n_nodes = len(off) - 1
    src = None if sources is None else _c(sources, np.int32)
    ns = n_nodes if src is None else len(src)
    idx = np.empty((ns, T), np.int32)
    cnt = np.empty((ns, T), np.uint16)
    wts = np.empty((ns, T), np.float32)
    steps = np.zeros(1, np.int64)
    lib.orc_build_neighborhoods(_ptr(off), _ptr(cl), num_pins, n_nodes, seed, walks, hops, T,
                                _ptr(src), ns, _ptr(idx), _ptr(cnt), _ptr(wts), _ptr(steps),
                                nthreads or default_threads())
    return idx, cnt, wts, int(steps[0])


def graph_neighborhoods(offsets, col, seed, T, sources=None, nthreads=None):
    """Sec. 3.4 MapReduce neighbourhoods: each node's CSR row (sampled with T
    draws when longer than T), distinct ids ascending with multiplicities and
    weights multiplicity / kept entries: (idx int32, counts uint16, weights fp32)."""
    lib = _load()
    off = _c(offsets, np.int64)
    cl = _c(col, np.int32)
    n_nodes = len(off) - 1
    src = None if sources is None else _c(sources, np.int32)
    ns = n_nodes if src is None else len(src)
    idx = np.empty((ns, T), np.int32)
    cnt = np.empty((ns, T), np.uint16)
    wts = np.empty((ns, T), np.float32)
    lib.orc_graph_neighborhoods(_ptr(off), _ptr(cl), n_nodes, seed, T, _ptr(src), ns, _ptr(idx),
                                _ptr(cnt), _ptr(wts), nthreads or default_threads())
    return idx, cnt, wts


def embed_all_bipartite(x_pins, num_nodes, layers, idx, wts, nthreads=None):
    """Sec. 3.4 MapReduce inference on the bipartite graph: boards have no
    features (h^(0) of a board is the zero vector), every node may be a
    neighbour, so all rows are projected at each layer; K layers, layer-wise."""
    xp = _c(x_pins, np.float64)
    h = np.zeros((num_nodes, xp.shape[1]), np.float64)
    h[: xp.shape[0]] = xp
    for L in layers:
        h = convolve_layer(h, num_nodes, L["Q"], L["q"], L["W"], L["w"], idx, wts,
                           nthreads=nthreads, pool=L.get("pool", "importance"))
    return h


POOLS = {"importance": 0, "mean": 1, "max": 2}


def convolve_layer(h_in, n_transform, Q, q, W, w, idx, wts, self_rows=None, nthreads=None,
                   pool="importance"):
    """One CONVOLVE layer (Algorithm 1) in the layer-wise dataflow of Sec. 3.4, fp64;
    `pool` is the aggregator gamma (importance, mean or max)."""
    lib = _load()
    h = _c(h_in, np.float64)
    Qd, qd, Wd, wd = _c(Q, np.float64), _c(q, np.float64), _c(W, np.float64), _c(w, np.float64)
    m, d_in = Qd.shape
    d_out = Wd.shape[0]
    assert Wd.shape[1] == d_in + m and h.shape[1] == d_in
    ix = _c(idx, np.int32)
    wt = _c(wts, np.float32)
    n_out, T = ix.shape
    sr = None if self_rows is None else _c(self_rows, np.int64)
    out = np.empty((n_out, d_out), np.float64)
    lib.orc_convolve_layer(_ptr(h), h.shape[0], d_in, n_transform, _ptr(Qd), _ptr(qd), m,
                           _ptr(Wd), _ptr(wd), d_out, _ptr(ix), _ptr(wt), T, _ptr(sr), n_out,
                           _ptr(out), nthreads or default_threads(), POOLS[pool])
    return out


def embed_all(x, num_pins, layers, idx, wts, nthreads=None):
    """K stacked layers over every node, layer-wise (Sec. 3.4): pins are the only
    neighbours, so rows [0, num_pins) are projected at each layer."""
    h = _c(x, np.float64)
    for L in layers:
        h = convolve_layer(h, num_pins, L["Q"], L["q"], L["W"], L["w"], idx, wts,
                           nthreads=nthreads, pool=L.get("pool", "importance"))
    return h


def minibatch_sets(targets, K, nbr_idx):
    """Algorithm 2 sampling: [S^(0), ..., S^(K)] as sorted int32 arrays."""
    lib = _load()
    tg = _c(targets, np.int32)
    ix = _c(nbr_idx, np.int32)
    T = ix.shape[1]
    sizes = np.zeros(K + 1, np.int64)
    need = lib.orc_minibatch_sets(_ptr(tg), len(tg), K, _ptr(ix), T, _ptr(sizes), None, 0)
    need = -need if need < 0 else need
    buf = np.empty(max(1, need), np.int32)
    got = lib.orc_minibatch_sets(_ptr(tg), len(tg), K, _ptr(ix), T, _ptr(sizes), _ptr(buf), need)
    assert got == need
    out, pos = [], 0
    for k in range(K + 1):
        out.append(buf[pos:pos + sizes[k]].copy())
        pos += sizes[k]
    return out


def minibatch_embed(targets, x, layers, nbr_idx, nbr_w, nthreads=None):
    """Algorithm 2 embedding loop for the targets (fp64); returns h^(K) per target."""
    lib = _load()
    tg = _c(targets, np.int32)
    xd = _c(x, np.float64)
    ix = _c(nbr_idx, np.int32)
    wt = _c(nbr_w, np.float32)
    K = len(layers)
    keep = []
    Qp, qp, Wp, wp = (ctypes.c_void_p * K)(), (ctypes.c_void_p * K)(), \
        (ctypes.c_void_p * K)(), (ctypes.c_void_p * K)()
    ms = np.zeros(K, np.int32)
    ds = np.zeros(K, np.int32)
    for k, L in enumerate(layers):
        Q, q, W, w = (_c(L[n], np.float64) for n in ("Q", "q", "W", "w"))
        keep += [Q, q, W, w]
        Qp[k], qp[k], Wp[k], wp[k] = (a.ctypes.data for a in (Q, q, W, w))
        ms[k] = Q.shape[0]
        ds[k] = W.shape[0]
    out = np.empty((len(tg), int(ds[-1])), np.float64)
    pools = _pools(layers)
    lib.orc_minibatch_embed(_ptr(tg), len(tg), K, _ptr(xd), xd.shape[1], _ptr(ix), _ptr(wt),
                            ix.shape[1], Qp, qp, _ptr(ms), Wp, wp, _ptr(ds), _ptr(out),
                            nthreads or default_threads(), _ptr(pools))
    return out


def _pools(layers):
    return np.array([POOLS[L.get("pool", "importance")] for L in layers], np.int32)


def _layer_ptrs(layers):
    K = len(layers)
    keep = []
    Qp, qp, Wp, wp = (ctypes.c_void_p * K)(), (ctypes.c_void_p * K)(), \
        (ctypes.c_void_p * K)(), (ctypes.c_void_p * K)()
    ms = np.zeros(K, np.int32)
    ds = np.zeros(K, np.int32)
    for k, L in enumerate(layers):
        Q, q, W, w = (_c(L[n], np.float64) for n in ("Q", "q", "W", "w"))
        keep += [Q, q, W, w]
        Qp[k], qp[k], Wp[k], wp[k] = (a.ctypes.data for a in (Q, q, W, w))
        ms[k] = Q.shape[0]
        ds[k] = W.shape[0]
    return keep, Qp, qp, Wp, wp, ms, ds


def minibatch_sample(targets, K, offsets, col, num_pins, seed, walks, hops, T, nthreads=None):
    """Algorithm 2 sampling with neighbourhoods computed on demand (Sec. 3.2 walks
    for each needed node only). Returns {"sets": [S^(0..K)], "row_ids", "idx", "wts"}
    with one neighbourhood row (sorted by node id) for every node of S^(1)."""
    lib = _load()
    tg = _c(targets, np.int32)
    off = _c(offsets, np.int64)
    cl = _c(col, np.int32)
    h = lib.orc_minibatch_sample(_ptr(tg), len(tg), K, _ptr(off), _ptr(cl), num_pins,
                                 len(off) - 1, seed, walks, hops, T, nthreads or default_threads())
    try:
        sizes = np.zeros(K + 2, np.int64)
        lib.orc_sample_sizes(h, K, _ptr(sizes))
        sets = np.empty(int(sizes[:K + 1].sum()), np.int32)
        nrow = int(sizes[K + 1])
        row_ids = np.empty(nrow, np.int32)
        idx = np.empty((nrow, T), np.int32)
        wts = np.empty((nrow, T), np.float32)
        lib.orc_sample_copy(h, K, _ptr(sets), _ptr(row_ids), _ptr(idx), _ptr(wts))
    finally:
        lib.orc_sample_free(h)
    out, pos = [], 0
    for k in range(K + 1):
        out.append(sets[pos:pos + sizes[k]])
        pos += sizes[k]
    return {"sets": out, "row_ids": row_ids, "idx": idx, "wts": wts}


def minibatch_embed_sampled(targets, x_ids, x_rows, sample, layers, nthreads=None):
    """Algorithm 2 embedding loop (fp64) from a sample: x_rows[i] is the feature
    row of node x_ids[i] (sorted ids covering S^(0))."""
    lib = _load()
    tg = _c(targets, np.int32)
    xi = _c(x_ids, np.int32)
    xr = _c(x_rows, np.float64)
    keep, Qp, qp, Wp, wp, ms, ds = _layer_ptrs(layers)
    out = np.empty((len(tg), int(ds[-1])), np.float64)
    ri, ix, wt = (_c(sample["row_ids"], np.int32), _c(sample["idx"], np.int32),
                  _c(sample["wts"], np.float32))
    lib.orc_minibatch_embed_sampled(_ptr(tg), len(tg), len(layers), _ptr(xi), len(xi), _ptr(xr),
                                    xr.shape[1], _ptr(ri), len(ri), _ptr(ix), _ptr(wt),
                                    ix.shape[1], Qp, qp, _ptr(ms), Wp, wp, _ptr(ds), _ptr(out),
                                    nthreads or default_threads(), _ptr(_pools(layers)))
    return out


def output_mlp(h, G1, g, G2, nthreads=None):
    """Algorithm 2's final dense layers, z = G2 ReLU(G1 h + g), per row (fp64)."""
    lib = _load()
    hd = _c(h, np.float64)
    A, b, B = _c(G1, np.float64), _c(g, np.float64), _c(G2, np.float64)
    d_hidden, d_in = A.shape
    d_out = B.shape[0]
    assert hd.shape[1] == d_in and B.shape[1] == d_hidden and b.shape == (d_hidden,)
    z = np.empty((hd.shape[0], d_out), np.float64)
    lib.orc_output_mlp(_ptr(hd), hd.shape[0], d_in, _ptr(A), _ptr(b), d_hidden, _ptr(B), d_out,
                       _ptr(z), nthreads or default_threads())
    return z


def max_margin_loss(zq, zpos, zneg, margin, zhard=None, hard_valid=None):
    """Eq. (1) with the expectation read as the mean over the shared negatives,
    joined per pair by its hard negatives zhard[b] ([B][k][d]; hard_valid[b][j]
    false drops an entry); returns (minibatch mean loss, per-pair terms)."""
    lib = _load()
    a, b, c = _c(zq, np.float64), _c(zpos, np.float64), _c(zneg, np.float64)
    per = np.empty(a.shape[0], np.float64)
    if zhard is None:
        loss = lib.orc_max_margin_loss(_ptr(a), _ptr(b), a.shape[0], _ptr(c), c.shape[0],
                                       a.shape[1], margin, _ptr(per))
        return float(loss), per
    h = _c(zhard, np.float64)
    B, k = h.shape[0], h.shape[1]
    assert B == a.shape[0] and h.shape[2] == a.shape[1]
    v = _c(np.ones((B, k), bool) if hard_valid is None else hard_valid, np.uint8)
    loss = lib.orc_max_margin_loss_hard(_ptr(a), _ptr(b), B, _ptr(c), c.shape[0], _ptr(h),
                                        _ptr(v), k, a.shape[1], margin, _ptr(per))
    return float(loss), per


def hard_negatives(offsets, col, num_pins, seed, walks, hops, queries, rank_lo, rank_hi, k,
                   nthreads=None):
    """Sec. 3.3 hard negatives: k pins per query drawn from the PPR rank window
    [rank_lo, rank_hi) (visit-count ranking of the query's own walks); -1 where
    the window is empty."""
    lib = _load()
    off = _c(offsets, np.int64)
    cl = _c(col, np.int32)
    q = _c(queries, np.int32)
    out = np.empty((len(q), k), np.int32)
    lib.orc_hard_negatives(_ptr(off), _ptr(cl), num_pins, len(off) - 1, seed, walks, hops,
                           _ptr(q), len(q), rank_lo, rank_hi, k, _ptr(out),
                           nthreads or default_threads())
    return out
