"""Python binding of libpinsage.so.

Argument marshalling only: PyTorch provides device memory and the current HIP
stream; every step of the hot path runs in the library's gfx950 kernels. The
functions mirror the C entry points of include/pinsage.h.
"""

from __future__ import annotations

import ctypes
from dataclasses import dataclass
from typing import List, Optional, Sequence

import numpy as np
import torch

from . import _lib as L


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream: Optional[torch.cuda.Stream]):
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _dev(t: torch.Tensor, name: str, dtype=None) -> torch.Tensor:
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise ValueError(f"{name} must be a CUDA (HIP) tensor")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} must have dtype {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t


def _dtype_code(dt: torch.dtype) -> int:
    if dt == torch.float32:
        return L.PINSAGE_F32
    if dt == torch.bfloat16:
        return L.PINSAGE_BF16
    raise ValueError(f"storage dtype must be float32 or bfloat16, got {dt}")


class DeviceGraph:
    """Bipartite pin-board CSR resident on the GPU (pins [0, P), boards [P, P+B))."""

    def __init__(self, offsets, col, num_pins: int, num_boards: int, device="cuda",
                 offsets64: Optional[bool] = None):
        if not torch.is_tensor(offsets):
            offsets = torch.as_tensor(np.asarray(offsets))
        if not torch.is_tensor(col):
            col = torch.as_tensor(np.asarray(col))
        nnz = int(col.numel())
        if offsets64 is None:
            offsets64 = nnz >= 2**31
        self.num_pins, self.num_boards, self.nnz = int(num_pins), int(num_boards), nnz
        self.offsets64 = bool(offsets64)
        odt = torch.int64 if self.offsets64 else torch.int32
        self.offsets = offsets.to(device=device, dtype=odt).contiguous()
        self.col = col.to(device=device, dtype=torch.int32).contiguous()
        self.walk_table: Optional[torch.Tensor] = None
        if self.offsets.numel() != self.num_nodes + 1:
            raise ValueError("offsets must have num_nodes + 1 entries")

    @property
    def num_nodes(self) -> int:
        return self.num_pins + self.num_boards

    def build_walk_table(self, stream=None) -> "DeviceGraph":
        """Builds the graph's walk table (16 bytes per CSR position); every later
        walk on this graph reads it (same results, one read per edge step)."""
        n = ctypes.c_size_t(0)
        self.walk_table = None
        L.check(L.lib().pinsage_walk_table_size(ctypes.byref(self.struct()), ctypes.byref(n)),
                "pinsage_walk_table_size")
        table = torch.empty(max(1, n.value), dtype=torch.uint8, device=self.col.device)
        L.check(L.lib().pinsage_build_walk_table(ctypes.byref(self.struct()), table.data_ptr(),
                                                 table.numel(), _stream(stream)),
                "pinsage_build_walk_table")
        self.walk_table = table
        return self

    def drop_walk_table(self) -> None:
        self.walk_table = None

    def struct(self) -> L.Graph:
        return L.Graph(self.num_pins, self.num_boards, self.nnz,
                       L.PINSAGE_I64 if self.offsets64 else L.PINSAGE_I32,
                       self.offsets.data_ptr(), self.col.data_ptr(),
                       self.walk_table.data_ptr() if self.walk_table is not None else None)


@dataclass
class Neighborhoods:
    idx: torch.Tensor       # int32 [rows, T]
    counts: torch.Tensor    # uint16 [rows, T]
    weights: Optional[torch.Tensor]  # float32 [rows, T]

    @property
    def rows(self) -> int:
        return int(self.idx.shape[0])

    @property
    def top_t(self) -> int:
        return int(self.idx.shape[1])

    def struct(self) -> L.Neighborhoods:
        return L.Neighborhoods(self.rows, self.top_t, self.idx.data_ptr(), self.counts.data_ptr(),
                               self.weights.data_ptr() if self.weights is not None else None)

    @staticmethod
    def empty(rows: int, T: int, weights: bool = True, device="cuda") -> "Neighborhoods":
        return Neighborhoods(torch.empty((rows, T), dtype=torch.int32, device=device),
                             torch.empty((rows, T), dtype=torch.uint16, device=device),
                             torch.empty((rows, T), dtype=torch.float32, device=device)
                             if weights else None)


class DeviceLayer:
    """One CONVOLVE layer's parameters on the GPU: Q [m, d_in], q [m] fp32,
    W [d_out, d_in + m], w [d_out] fp32; Q and W in the storage dtype.

    dataflow: "pool_then_dense" (Algorithm 1 as written: pool m-wide
    transformed rows, then W) or "dense_then_pool" (the neighbour half of W is
    applied per pin first, so the pool gathers d_out-wide rows); both compute
    the same layer. pool: the aggregator gamma, "importance" (Sec. 3.2), "mean"
    or "max" (Sec. 4); "max" needs "pool_then_dense"."""

    def __init__(self, Q, q, W, w, dtype: torch.dtype = torch.float32, device="cuda",
                 dataflow: str = "pool_then_dense", pool: str = "importance"):
        if dataflow not in L.DATAFLOWS:
            raise ValueError(f"dataflow must be one of {sorted(L.DATAFLOWS)}, got {dataflow!r}")
        if pool not in L.POOLS:
            raise ValueError(f"pool must be one of {sorted(L.POOLS)}, got {pool!r}")
        self.dataflow = dataflow
        self.pool = pool
        self.dtype = dtype
        self.Q = torch.as_tensor(Q).to(device=device, dtype=dtype).contiguous()
        self.W = torch.as_tensor(W).to(device=device, dtype=dtype).contiguous()
        self.q = torch.as_tensor(q).to(device=device, dtype=torch.float32).contiguous()
        self.w = torch.as_tensor(w).to(device=device, dtype=torch.float32).contiguous()
        self.m, self.d_in = self.Q.shape
        self.d_out = self.W.shape[0]
        if self.W.shape[1] != self.d_in + self.m:
            raise ValueError("W must be [d_out, d_in + m]")

    def struct(self) -> L.Layer:
        return L.Layer(self.d_in, self.m, self.d_out, _dtype_code(self.dtype), self.Q.data_ptr(),
                       self.q.data_ptr(), self.W.data_ptr(), self.w.data_ptr(),
                       L.DATAFLOWS[self.dataflow], L.POOLS[self.pool])


class DeviceMLP:
    """Output dense layers of Algorithm 2 on the GPU: z = G2 ReLU(G1 h + g);
    G1 [d_hidden, d_in], g [d_hidden] fp32, G2 [d_out, d_hidden]."""

    def __init__(self, G1, g, G2, dtype: torch.dtype = torch.float32, device="cuda"):
        self.dtype = dtype
        self.G1 = torch.as_tensor(G1).to(device=device, dtype=dtype).contiguous()
        self.G2 = torch.as_tensor(G2).to(device=device, dtype=dtype).contiguous()
        self.g = torch.as_tensor(g).to(device=device, dtype=torch.float32).contiguous()
        self.d_hidden, self.d_in = self.G1.shape
        self.d_out = self.G2.shape[0]
        if self.G2.shape[1] != self.d_hidden or self.g.numel() != self.d_hidden:
            raise ValueError("G2 must be [d_out, d_hidden] and g [d_hidden]")

    def struct(self) -> L.MLP:
        return L.MLP(self.d_in, self.d_hidden, self.d_out, _dtype_code(self.dtype),
                     self.G1.data_ptr(), self.g.data_ptr(), self.G2.data_ptr())


def output_mlp(mlp: DeviceMLP, h: torch.Tensor, out: Optional[torch.Tensor] = None,
               workspace: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """z = G2 ReLU(G1 h + g) for every row of h (Algorithm 2, final loop)."""
    h = _dev(h, "h", mlp.dtype)
    n = int(h.shape[0])
    if out is None:
        out = torch.empty((n, mlp.d_out), dtype=mlp.dtype, device=h.device)
    _dev(out, "out", mlp.dtype)
    m = mlp.struct()
    need = ctypes.c_size_t(0)
    L.check(L.lib().pinsage_output_mlp_workspace_size(ctypes.byref(m), n, ctypes.byref(need)),
            "pinsage_output_mlp_workspace_size")
    if workspace is None:
        workspace = torch.empty(max(1, int(need.value)), dtype=torch.uint8, device=h.device)
    L.check(L.lib().pinsage_output_mlp(ctypes.byref(m), _ptr(h), n, _ptr(out), _ptr(workspace),
                                       workspace.numel(), _stream(stream)),
            "pinsage_output_mlp")
    return out


def build_neighborhoods(graph: DeviceGraph, walks: int, hops: int, T: int, seed: int,
                        sources: Optional[torch.Tensor] = None, weights: bool = True,
                        out: Optional[Neighborhoods] = None, count_steps: bool = True,
                        stream=None):
    """Importance neighbourhoods (Sec. 3.2). Returns (Neighborhoods, total_steps tensor|None)."""
    lib = L.lib()
    if sources is not None:
        sources = _dev(sources, "sources", torch.int32)
    rows = graph.num_nodes if sources is None else int(sources.numel())
    nb = out if out is not None else Neighborhoods.empty(rows, T, weights, graph.col.device)
    steps = torch.empty(1, dtype=torch.int64, device=graph.col.device) if count_steps else None
    g, wp, ns = graph.struct(), L.WalkParams(seed, walks, hops, T), nb.struct()
    st = lib.pinsage_build_neighborhoods(ctypes.byref(g), ctypes.byref(wp), _ptr(sources), rows,
                                         ctypes.byref(ns), _ptr(steps), _stream(stream))
    L.check(st, "pinsage_build_neighborhoods")
    return nb, steps


def hard_negatives(graph: DeviceGraph, queries: torch.Tensor, k: int, seed: int, walks: int,
                   hops: int, rank_lo: int = 1999, rank_hi: int = 5000,
                   out: Optional[torch.Tensor] = None, count_steps: bool = False, stream=None):
    """Hard negative items (Sec. 3.3): k pins per query drawn from ranks
    [rank_lo, rank_hi) of the query's visit-count (PPR) ranking; -1 where the
    window is empty. Returns (out int32 [n][k], total_steps tensor|None)."""
    lib = L.lib()
    queries = _dev(queries, "queries", torch.int32)
    n = int(queries.numel())
    if out is None:
        out = torch.empty((n, k), dtype=torch.int32, device=queries.device)
    steps = torch.empty(1, dtype=torch.int64, device=queries.device) if count_steps else None
    g = graph.struct()
    hp = L.HardNegativeParams(seed, walks, hops, rank_lo, rank_hi, k)
    need = ctypes.c_size_t(0)
    L.check(lib.pinsage_hard_negatives_workspace_size(ctypes.byref(hp), n, ctypes.byref(need)),
            "pinsage_hard_negatives_workspace_size")
    ws = (torch.empty(int(need.value), dtype=torch.uint8, device=queries.device)
          if need.value else None)
    st = lib.pinsage_hard_negatives(ctypes.byref(g), ctypes.byref(hp), _ptr(queries), n, _ptr(out),
                                    _ptr(steps), _ptr(ws), int(need.value), _stream(stream))
    L.check(st, "pinsage_hard_negatives")
    return out, steps


def convolve_workspace_size(layer: DeviceLayer, n_transform: int, n_out: int) -> int:
    n = ctypes.c_size_t(0)
    st = L.lib().pinsage_convolve_workspace_size(ctypes.byref(layer.struct()), n_transform, n_out,
                                                 ctypes.byref(n))
    L.check(st, "pinsage_convolve_workspace_size")
    return int(n.value)


def convolve_layer(layer: DeviceLayer, h_in: torch.Tensor, n_transform: int, nbr: Neighborhoods,
                   self_rows: Optional[torch.Tensor] = None, out: Optional[torch.Tensor] = None,
                   workspace: Optional[torch.Tensor] = None, transform_rows=None,
                   stream=None) -> torch.Tensor:
    """One CONVOLVE layer (Algorithm 1) in the layer-wise dataflow (Sec. 3.4)."""
    lib = L.lib()
    h_in = _dev(h_in, "h_in", layer.dtype)
    if self_rows is not None:
        self_rows = _dev(self_rows, "self_rows", torch.int32)
    if transform_rows is not None:
        transform_rows = _dev(transform_rows, "transform_rows", torch.int32)
        n_transform = int(transform_rows.numel())
    n_out = nbr.rows
    if out is None:
        out = torch.empty((n_out, layer.d_out), dtype=layer.dtype, device=h_in.device)
    _dev(out, "out", layer.dtype)
    need = convolve_workspace_size(layer, n_transform, n_out)
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=h_in.device)
    ns = nbr.struct()
    st = lib.pinsage_convolve_layer(ctypes.byref(layer.struct()), _ptr(h_in), h_in.shape[0],
                                    n_transform, _ptr(transform_rows), ctypes.byref(ns),
                                    _ptr(self_rows), _ptr(out),
                                    n_out, _ptr(workspace), workspace.numel(), _stream(stream))
    L.check(st, "pinsage_convolve_layer")
    return out


def _layer_array(layers: Sequence[DeviceLayer]):
    arr = (L.Layer * len(layers))()
    for i, ly in enumerate(layers):
        arr[i] = ly.struct()
    return arr


def embed_all_workspace_size(graph: DeviceGraph, layers: Sequence[DeviceLayer]) -> int:
    n = ctypes.c_size_t(0)
    st = L.lib().pinsage_embed_all_workspace_size(ctypes.byref(graph.struct()),
                                                  _layer_array(layers), len(layers),
                                                  ctypes.byref(n))
    L.check(st, "pinsage_embed_all_workspace_size")
    return int(n.value)


class Schedule:
    """A caller-owned schedule of the all-node job (pinsage_schedule_t): two
    CU-masked streams of the current device, on which the walks and the first
    layer's transform of a leading share of the pins run beside each other
    (the transform on cu_eighths / 8 of the CUs). close() waits for them and
    destroys them; so does garbage collection."""

    def __init__(self, cu_eighths: int):
        h = ctypes.c_void_p(None)
        L.check(L.lib().pinsage_schedule_create(int(cu_eighths), ctypes.byref(h)),
                "pinsage_schedule_create")
        self.cu_eighths = int(cu_eighths)
        self.handle = h.value

    def close(self) -> None:
        h, self.handle = getattr(self, "handle", None), None
        if h:
            L.check(L.lib().pinsage_schedule_destroy(h), "pinsage_schedule_destroy")

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class EmbedAll:
    """Preallocated all-node embedding job (neighbourhoods + K layers, Sec. 3.4).
    overlap: 0 runs the walks and the first transform in order; 1-7 gives the
    job a Schedule on that many eighths of the CUs (used for graphs of 2^18 to
    2^22 pins, and above 2^22 when the first layer is chained and the walk
    table fits in the first layer's output buffer; the output is the same bits
    either way)."""

    def __init__(self, graph: DeviceGraph, layers: List[DeviceLayer], walks: int, hops: int,
                 T: int, seed: int, weights: bool = True, overlap: int = 0):
        self.graph, self.layers = graph, list(layers)
        self.walk = L.WalkParams(seed, walks, hops, T)
        dev = graph.col.device
        self.nbr = Neighborhoods.empty(graph.num_nodes, T, weights, dev)
        self.out = torch.empty((graph.num_nodes, layers[-1].d_out), dtype=layers[-1].dtype,
                               device=dev)
        self.steps = torch.zeros(1, dtype=torch.int64, device=dev)
        self.workspace = torch.empty(max(1, embed_all_workspace_size(graph, layers)),
                                     dtype=torch.uint8, device=dev)
        self._g = graph.struct()
        self._layers = _layer_array(self.layers)
        self._nbr = self.nbr.struct()
        self.schedule = Schedule(overlap) if overlap else None

    def run(self, x: torch.Tensor, stream=None) -> torch.Tensor:
        x = _dev(x, "x", self.layers[0].dtype)
        sched = self.schedule.handle if self.schedule is not None else None
        self._g = self.graph.struct()  # picks up a walk table built since
        st = L.lib().pinsage_embed_all(ctypes.byref(self._g), ctypes.byref(self.walk),
                                       self._layers, len(self.layers), _ptr(x),
                                       ctypes.byref(self._nbr), _ptr(self.out), _ptr(self.steps),
                                       _ptr(self.workspace), self.workspace.numel(), sched,
                                       _stream(stream))
        L.check(st, "pinsage_embed_all")
        return self.out

    def close(self) -> None:
        if self.schedule is not None:
            self.schedule.close()
            self.schedule = None


def build_graph_neighborhoods(graph: DeviceGraph, T: int, seed: int,
                              sources: Optional[torch.Tensor] = None, weights: bool = True,
                              out: Optional[Neighborhoods] = None, stream=None) -> Neighborhoods:
    """Graph neighbourhoods of the MapReduce inference (Sec. 3.4): CSR rows, or
    T Philox draws from rows longer than T, distinct ids ascending."""
    if sources is not None:
        sources = _dev(sources, "sources", torch.int32)
    rows = graph.num_nodes if sources is None else int(sources.numel())
    nb = out if out is not None else Neighborhoods.empty(rows, T, weights, graph.col.device)
    g, ns = graph.struct(), nb.struct()
    st = L.lib().pinsage_build_graph_neighborhoods(ctypes.byref(g), seed, _ptr(sources), rows,
                                                   ctypes.byref(ns), _stream(stream))
    L.check(st, "pinsage_build_graph_neighborhoods")
    return nb


class EmbedAllBipartite:
    """Preallocated all-node job of the MapReduce inference (Sec. 3.4): graph
    neighbourhoods, then an even number of layers over all nodes with
    featureless boards; x holds the pins' features only."""

    def __init__(self, graph: DeviceGraph, layers: List[DeviceLayer], T: int, seed: int,
                 weights: bool = True):
        self.graph, self.layers, self.seed = graph, list(layers), int(seed)
        dev = graph.col.device
        self.nbr = Neighborhoods.empty(graph.num_nodes, T, weights, dev)
        self.out = torch.empty((graph.num_nodes, layers[-1].d_out), dtype=layers[-1].dtype,
                               device=dev)
        self._g = graph.struct()
        self._layers = _layer_array(self.layers)
        self._nbr = self.nbr.struct()
        n = ctypes.c_size_t(0)
        st = L.lib().pinsage_embed_all_bipartite_workspace_size(ctypes.byref(self._g),
                                                                self._layers, len(self.layers),
                                                                ctypes.byref(n))
        L.check(st, "pinsage_embed_all_bipartite_workspace_size")
        self.workspace = torch.empty(max(1, int(n.value)), dtype=torch.uint8, device=dev)

    def run(self, x_pins: torch.Tensor, stream=None) -> torch.Tensor:
        x = _dev(x_pins, "x_pins", self.layers[0].dtype)
        if x.shape[0] != self.graph.num_pins:
            raise ValueError("x_pins must have one row per pin")
        st = L.lib().pinsage_embed_all_bipartite(ctypes.byref(self._g), self.seed, self._layers,
                                                 len(self.layers), _ptr(x),
                                                 ctypes.byref(self._nbr), _ptr(self.out),
                                                 _ptr(self.workspace), self.workspace.numel(),
                                                 _stream(stream))
        L.check(st, "pinsage_embed_all_bipartite")
        return self.out


def embed_all(graph: DeviceGraph, layers: List[DeviceLayer], x: torch.Tensor, walks: int,
              hops: int, T: int, seed: int, stream=None):
    job = EmbedAll(graph, layers, walks, hops, T, seed)
    out = job.run(x, stream)
    return job.nbr, out, job.steps


def max_margin_loss(zq: torch.Tensor, zpos: torch.Tensor, zneg: torch.Tensor, margin: float,
                    zhard: Optional[torch.Tensor] = None, stream=None):
    """Eq. (1) with the mean over the shared negatives joined by each pair's
    hard negatives zhard[b] ([B][k][d], optional); returns (loss, per_pair)."""
    dt = zq.dtype
    for t, n in ((zq, "zq"), (zpos, "zpos"), (zneg, "zneg")):
        _dev(t, n, dt)
    B, d = zq.shape
    k = 0
    if zhard is not None:
        _dev(zhard, "zhard", dt)
        if zhard.dim() != 3 or zhard.shape[0] != B or zhard.shape[2] != d:
            raise ValueError("zhard must be [B][k][d]")
        k = int(zhard.shape[1])
    loss = torch.empty(1, dtype=torch.float32, device=zq.device)
    per = torch.empty(B, dtype=torch.float32, device=zq.device)
    st = L.lib().pinsage_max_margin_loss(_ptr(zq), _ptr(zpos), B, _ptr(zneg), zneg.shape[0],
                                         _ptr(zhard), k, d, _dtype_code(dt), margin, _ptr(loss),
                                         _ptr(per), _stream(stream))
    L.check(st, "pinsage_max_margin_loss")
    return loss, per


class Minibatch:
    """Minibatch forward of Algorithm 2 plus the loss of Eq. (1), with a
    preallocated workspace sized for num_pairs pairs, num_negatives shared
    negatives and num_hard hard negatives per pair."""

    def __init__(self, graph: DeviceGraph, layers: List[DeviceLayer], walks: int, hops: int,
                 T: int, seed: int, num_pairs: int, num_negatives: int,
                 mlp: Optional[DeviceMLP] = None, num_hard: int = 0):
        self.graph, self.layers = graph, list(layers)
        self.mlp = mlp
        self._mlp = mlp.struct() if mlp is not None else None
        self.walk = L.WalkParams(seed, walks, hops, T)
        self.B, self.n_neg, self.k_hard = int(num_pairs), int(num_negatives), int(num_hard)
        self._g = graph.struct()
        self._layers = _layer_array(self.layers)
        n = ctypes.c_size_t(0)
        st = L.lib().pinsage_minibatch_workspace_size(ctypes.byref(self._g), ctypes.byref(self.walk),
                                                      self._layers, len(self.layers),
                                                      self._mlp_ref(), self.B, self.n_neg,
                                                      self.k_hard, ctypes.byref(n))
        L.check(st, "pinsage_minibatch_workspace_size")
        dev = graph.col.device
        self.workspace = torch.empty(max(1, int(n.value)), dtype=torch.uint8, device=dev)
        self.loss = torch.empty(1, dtype=torch.float32, device=dev)
        self.per_pair = torch.empty(self.B, dtype=torch.float32, device=dev)
        d = mlp.d_out if mlp is not None else self.layers[-1].d_out
        self.z = torch.empty((2 * self.B + self.n_neg + self.B * self.k_hard, d),
                             dtype=self.layers[-1].dtype, device=dev)
        self.set_sizes = (ctypes.c_int64 * (len(self.layers) + 1))()
        self.steps = torch.zeros(1, dtype=torch.int64, device=dev)  # edge steps of the last run

    def run(self, x: torch.Tensor, queries: torch.Tensor, positives: torch.Tensor,
            negatives: torch.Tensor, margin: float, want_z: bool = True,
            hard: Optional[torch.Tensor] = None, stream=None):
        """hard: int32 [num_pairs][num_hard] hard negatives (-1 = absent), required
        when the workspace was made for num_hard > 0."""
        x = _dev(x, "x", self.layers[0].dtype)
        q = _dev(queries, "queries", torch.int32)
        p = _dev(positives, "positives", torch.int32)
        ng = _dev(negatives, "negatives", torch.int32)
        if q.numel() != self.B or p.numel() != self.B or ng.numel() != self.n_neg:
            raise ValueError("pair counts differ from the sizes this workspace was made for")
        hp = None
        if self.k_hard:
            if hard is None or hard.numel() != self.B * self.k_hard:
                raise ValueError(f"hard must hold num_pairs x {self.k_hard} ids")
            hp = _dev(hard, "hard", torch.int32).data_ptr()
        pairs = L.Pairs(self.B, self.n_neg, q.data_ptr(), p.data_ptr(), ng.data_ptr(), margin,
                        self.k_hard, hp)
        self._g = self.graph.struct()  # picks up a walk table built since
        st = L.lib().pinsage_minibatch_forward(ctypes.byref(self._g), ctypes.byref(self.walk),
                                               self._layers, len(self.layers), self._mlp_ref(),
                                               _ptr(x),
                                               ctypes.byref(pairs), _ptr(self.loss),
                                               _ptr(self.per_pair),
                                               _ptr(self.z) if want_z else None, self.set_sizes,
                                               _ptr(self.steps), _ptr(self.workspace),
                                               self.workspace.numel(),
                                               _stream(stream))
        L.check(st, "pinsage_minibatch_forward")
        return self.loss

    def sizes(self) -> list:
        return [int(v) for v in self.set_sizes]

    def _mlp_ref(self):
        return ctypes.byref(self._mlp) if self._mlp is not None else None


def profile_enable(on: bool = True) -> None:
    L.check(L.lib().pinsage_profile_enable(1 if on else 0), "pinsage_profile_enable")


def profile_read() -> dict:
    """{kernel name: (launches, total ms)} for launches timed since profile_enable."""
    out = {}
    for k, name in enumerate(L.KERNEL_NAMES):
        n = ctypes.c_int64(0)
        ms = ctypes.c_double(0)
        L.check(L.lib().pinsage_profile_read(k, ctypes.byref(n), ctypes.byref(ms)),
                "pinsage_profile_read")
        out[name] = (int(n.value), float(ms.value))
    return out
