"""Seeded synthetic inputs for the PinSage hot path.

This module only draws inputs: a bipartite pin-board graph in CSR form, node
features and layer (and output-layer) parameters. It holds none of the method's arithmetic
(no walks, no pooling, no layers), so both the GPU library's tests and the CPU
oracle can consume the same inputs without sharing any computation.

Workload shapes follow the paper's setting (Sec. 3.1: pins and boards form a
bipartite graph, pins carry real-valued features) at sizes one GPU holds.
"""

from .graphs import (  # noqa: F401
    Workload,
    WORKLOADS,
    make_graph,
    make_layers,
    make_mlp,
    make_features,
    make_workload,
    bf16_round,
    csr_from_edges,
    minibatch_pairs,
    random_neighborhoods,
)
