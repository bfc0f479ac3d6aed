"""ctypes view of libpinsage.so (declarations mirror include/pinsage.h)."""

from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libpinsage.so")

PINSAGE_OK = 0
PINSAGE_EINVAL = -1
PINSAGE_EUNSUPPORTED = -2
PINSAGE_EWORKSPACE = -3
PINSAGE_EHIP = -4

PINSAGE_I32, PINSAGE_I64 = 0, 1
PINSAGE_F32, PINSAGE_BF16 = 0, 1
PINSAGE_POOL_THEN_DENSE, PINSAGE_DENSE_THEN_POOL = 0, 1
DATAFLOWS = {"pool_then_dense": PINSAGE_POOL_THEN_DENSE, "dense_then_pool": PINSAGE_DENSE_THEN_POOL}
POOLS = {"importance": 0, "mean": 1, "max": 2}

(KERNEL_WALK, KERNEL_GEMM_Q, KERNEL_POOL, KERNEL_GEMM_W, KERNEL_MINIBATCH, KERNEL_LOSS,
 KERNEL_GEMM_R, KERNEL_MLP) = range(8)
KERNEL_NAMES = ["walk_topt", "gemm_q", "pool", "gemm_w", "minibatch", "loss", "gemm_r", "mlp",
                "hard_neg", "graph_nbr", "gemm_qr", "walk_table",
                "pool_w"]

EXPORTED = [
    "pinsage_version", "pinsage_status_string", "pinsage_last_error",
    "pinsage_build_neighborhoods", "pinsage_hard_negatives",
    "pinsage_hard_negatives_workspace_size", "pinsage_build_graph_neighborhoods",
    "pinsage_embed_all_bipartite_workspace_size", "pinsage_embed_all_bipartite",
    "pinsage_convolve_workspace_size", "pinsage_convolve_layer", "pinsage_convolve_layer_noalloc",
    "pinsage_embed_all_workspace_size", "pinsage_embed_all",
    "pinsage_schedule_create", "pinsage_schedule_destroy",
    "pinsage_output_mlp_workspace_size",
    "pinsage_output_mlp", "pinsage_max_margin_loss",
    "pinsage_minibatch_workspace_size", "pinsage_minibatch_forward",
    "pinsage_profile_enable", "pinsage_profile_read", "pinsage_profile_random_reads",
    "pinsage_profile_random_gathers", "pinsage_walk_table_size", "pinsage_build_walk_table",
]


class Graph(ctypes.Structure):
    _fields_ = [("num_pins", ctypes.c_int64), ("num_boards", ctypes.c_int64),
                ("nnz", ctypes.c_int64), ("offset_type", ctypes.c_int),
                ("row_offsets", ctypes.c_void_p), ("col", ctypes.c_void_p),
                ("walk_table", ctypes.c_void_p)]


class WalkParams(ctypes.Structure):
    _fields_ = [("seed", ctypes.c_uint64), ("walks_per_node", ctypes.c_int32),
                ("hops", ctypes.c_int32), ("top_t", ctypes.c_int32)]


class Neighborhoods(ctypes.Structure):
    _fields_ = [("rows", ctypes.c_int64), ("top_t", ctypes.c_int32),
                ("idx", ctypes.c_void_p), ("counts", ctypes.c_void_p),
                ("weights", ctypes.c_void_p)]


class Layer(ctypes.Structure):
    _fields_ = [("d_in", ctypes.c_int32), ("m", ctypes.c_int32), ("d_out", ctypes.c_int32),
                ("dtype", ctypes.c_int), ("Q", ctypes.c_void_p), ("q", ctypes.c_void_p),
                ("W", ctypes.c_void_p), ("w", ctypes.c_void_p), ("dataflow", ctypes.c_int),
                ("pool", ctypes.c_int)]


class HardNegativeParams(ctypes.Structure):
    _fields_ = [("seed", ctypes.c_uint64), ("walks", ctypes.c_int32), ("hops", ctypes.c_int32),
                ("rank_lo", ctypes.c_int32), ("rank_hi", ctypes.c_int32),
                ("num_per_query", ctypes.c_int32)]


class MLP(ctypes.Structure):
    _fields_ = [("d_in", ctypes.c_int32), ("d_hidden", ctypes.c_int32), ("d_out", ctypes.c_int32),
                ("dtype", ctypes.c_int), ("G1", ctypes.c_void_p), ("g", ctypes.c_void_p),
                ("G2", ctypes.c_void_p)]


class Pairs(ctypes.Structure):
    _fields_ = [("num_pairs", ctypes.c_int64), ("num_negatives", ctypes.c_int64),
                ("queries", ctypes.c_void_p), ("positives", ctypes.c_void_p),
                ("negatives", ctypes.c_void_p), ("margin", ctypes.c_float),
                ("num_hard", ctypes.c_int64), ("hard_negatives", ctypes.c_void_p)]


class PinsageError(RuntimeError):
    def __init__(self, status: int, where: str, detail: str):
        super().__init__(f"{where}: status {status} ({detail})")
        self.status = status


_lib = None


def lib():
    """Load libpinsage.so; fails loudly if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                           "`python -c 'import __graft_entry__ as g; g.build()'`")
    L = ctypes.CDLL(LIB_PATH)
    P, i64, i32, u64 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_uint64
    L.pinsage_version.restype = ctypes.c_int
    L.pinsage_status_string.argtypes = [ctypes.c_int]
    L.pinsage_status_string.restype = ctypes.c_char_p
    L.pinsage_last_error.restype = ctypes.c_char_p
    L.pinsage_build_neighborhoods.argtypes = [ctypes.POINTER(Graph), ctypes.POINTER(WalkParams),
                                              P, i64, ctypes.POINTER(Neighborhoods), P, P]
    L.pinsage_build_graph_neighborhoods.argtypes = [ctypes.POINTER(Graph), u64, P, i64,
                                                    ctypes.POINTER(Neighborhoods), P]
    L.pinsage_embed_all_bipartite_workspace_size.argtypes = [ctypes.POINTER(Graph),
                                                             ctypes.POINTER(Layer), i32,
                                                             ctypes.POINTER(ctypes.c_size_t)]
    L.pinsage_embed_all_bipartite.argtypes = [ctypes.POINTER(Graph), u64, ctypes.POINTER(Layer),
                                              i32, P, ctypes.POINTER(Neighborhoods), P, P,
                                              ctypes.c_size_t, P]
    L.pinsage_hard_negatives.argtypes = [ctypes.POINTER(Graph), ctypes.POINTER(HardNegativeParams),
                                         P, i64, P, P, P, ctypes.c_size_t, P]
    L.pinsage_hard_negatives_workspace_size.argtypes = [ctypes.POINTER(HardNegativeParams), i64,
                                                        ctypes.POINTER(ctypes.c_size_t)]
    L.pinsage_convolve_workspace_size.argtypes = [ctypes.POINTER(Layer), i64, i64,
                                                  ctypes.POINTER(ctypes.c_size_t)]
    L.pinsage_convolve_layer.argtypes = [ctypes.POINTER(Layer), P, i64, i64, P,
                                         ctypes.POINTER(Neighborhoods), P, P, i64, P,
                                         ctypes.c_size_t, P]
    L.pinsage_convolve_layer_noalloc.argtypes = [ctypes.POINTER(Layer), P, i64, i64, P,
                                                 ctypes.POINTER(Neighborhoods), P, P, i64, P]
    L.pinsage_embed_all_workspace_size.argtypes = [ctypes.POINTER(Graph), ctypes.POINTER(Layer),
                                                   i32, ctypes.POINTER(ctypes.c_size_t)]
    L.pinsage_embed_all.argtypes = [ctypes.POINTER(Graph), ctypes.POINTER(WalkParams),
                                    ctypes.POINTER(Layer), i32, P, ctypes.POINTER(Neighborhoods),
                                    P, P, P, ctypes.c_size_t, P, P]
    L.pinsage_schedule_create.argtypes = [i32, ctypes.POINTER(ctypes.c_void_p)]
    L.pinsage_schedule_destroy.argtypes = [P]
    L.pinsage_output_mlp_workspace_size.argtypes = [ctypes.POINTER(MLP), i64,
                                                    ctypes.POINTER(ctypes.c_size_t)]
    L.pinsage_output_mlp.argtypes = [ctypes.POINTER(MLP), P, i64, P, P, ctypes.c_size_t, P]
    L.pinsage_max_margin_loss.argtypes = [P, P, i64, P, i64, P, i64, i32, ctypes.c_int,
                                          ctypes.c_float, P, P, P]
    L.pinsage_minibatch_workspace_size.argtypes = [ctypes.POINTER(Graph),
                                                   ctypes.POINTER(WalkParams),
                                                   ctypes.POINTER(Layer), i32, ctypes.POINTER(MLP),
                                                   i64, i64, i64, ctypes.POINTER(ctypes.c_size_t)]
    L.pinsage_minibatch_forward.argtypes = [ctypes.POINTER(Graph), ctypes.POINTER(WalkParams),
                                            ctypes.POINTER(Layer), i32, ctypes.POINTER(MLP), P,
                                            ctypes.POINTER(Pairs),
                                            P, P, P, ctypes.POINTER(ctypes.c_int64), P, P,
                                            ctypes.c_size_t, P]
    L.pinsage_profile_enable.argtypes = [ctypes.c_int]
    L.pinsage_profile_read.argtypes = [ctypes.c_int, ctypes.POINTER(ctypes.c_int64),
                                       ctypes.POINTER(ctypes.c_double)]
    L.pinsage_profile_random_reads.argtypes = [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int32,
                                               ctypes.c_int32, ctypes.c_void_p, ctypes.c_int64,
                                               ctypes.c_void_p]
    L.pinsage_profile_random_gathers.argtypes = [ctypes.c_void_p, ctypes.c_size_t,
                                                 ctypes.c_int32, ctypes.c_int64, ctypes.c_int32,
                                                 ctypes.c_uint64, ctypes.c_void_p, ctypes.c_void_p]
    L.pinsage_walk_table_size.argtypes = [ctypes.POINTER(Graph), ctypes.POINTER(ctypes.c_size_t)]
    L.pinsage_build_walk_table.argtypes = [ctypes.POINTER(Graph), P, ctypes.c_size_t, P]
    for name in EXPORTED:
        fn = getattr(L, name)
        if fn.restype is None or fn.restype is ctypes.c_int:
            fn.restype = ctypes.c_int
    _lib = L
    return L


def check(status: int, where: str) -> None:
    if status != PINSAGE_OK:
        detail = lib().pinsage_last_error().decode(errors="replace")
        raise PinsageError(status, where, detail or
                           lib().pinsage_status_string(status).decode())
