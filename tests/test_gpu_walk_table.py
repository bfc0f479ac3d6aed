"""GPU: the all-node job's walks read the walk table (one 16-byte entry per
CSR position carrying the neighbour's id, degree and row start) where
pinsage_build_neighborhoods reads the CSR. Both must give the same
neighbourhood table bit for bit, step totals included, on graphs with dead
ends, isolated nodes, out-of-range column ids and malformed rows, for both
walk widths (two sources per wave up to 64 walks, one above) and int64 row
offsets (Sec. 3.2: the walk definition does not depend on the layout).
"""

import numpy as np
import pytest
import torch

import synth

pytestmark = pytest.mark.gpu


def _layers(d=64):
    import paper_1806_01973_amd as ps
    g = torch.Generator().manual_seed(0)
    Q = torch.randn(d, d, generator=g) * 0.1
    W = torch.randn(d, 2 * d, generator=g) * 0.1
    return [ps.DeviceLayer(Q, torch.zeros(d), W, torch.zeros(d), dtype=torch.float32)]


def _both(off, col, P, B, walks, hops, T, seed, offsets64=False):
    import paper_1806_01973_amd as ps
    g = ps.DeviceGraph(off, col, P, B, offsets64=offsets64)
    nb, steps = ps.build_neighborhoods(g, walks, hops, T, seed)
    layers = _layers()
    job = ps.EmbedAll(g, layers, walks, hops, T, seed)
    x = torch.randn(P + B, 64, device="cuda")
    job.run(x)
    torch.cuda.synchronize()
    csr = (nb.idx.cpu().numpy(), nb.counts.cpu().numpy(), nb.weights.cpu().numpy(),
           int(steps.item()))
    tab = (job.nbr.idx.cpu().numpy(), job.nbr.counts.cpu().numpy(),
           job.nbr.weights.cpu().numpy(), int(job.steps.item()))
    job.close()
    return csr, tab


def _assert_same(a, b, what):
    np.testing.assert_array_equal(a[0], b[0], err_msg=f"{what}: idx")
    np.testing.assert_array_equal(a[1], b[1], err_msg=f"{what}: counts")
    np.testing.assert_array_equal(a[2].view(np.uint32), b[2].view(np.uint32),
                                  err_msg=f"{what}: weights")
    assert a[3] == b[3], f"{what}: steps {a[3]} != {b[3]}"


@pytest.mark.parametrize("walks,hops,T", [(20, 3, 5), (64, 2, 16), (100, 3, 50)])
def test_dead_ends_and_isolated_nodes(walks, hops, T):
    P, B = 6, 4
    edges = [(0, 0), (1, 0), (2, 1), (3, 1), (3, 0)]  # pins 4, 5 and boards 2, 3 isolated
    off, col = synth.csr_from_edges(P, B, edges)
    print(f"[case] walk table, dead ends W={walks}", flush=True)
    csr, tab = _both(off, col, P, B, walks, hops, T, 3)
    _assert_same(csr, tab, "dead ends")
    assert np.all(tab[0][4] == -1)


@pytest.mark.parametrize("offsets64", [False, True])
@pytest.mark.parametrize("walks", [50, 200])
def test_corrupt_ids_and_rows(walks, offsets64):
    # The tiny workload graph with out-of-range neighbour ids (negative and past
    # the last node) and two malformed rows: one whose end precedes its start
    # and, for the last node, an end past nnz. Walks end at such an entry or
    # row on both paths.
    wl = synth.WORKLOADS["tiny"]
    off, col, _ = synth.make_graph(wl)
    off = np.asarray(off, np.int64).copy()
    col = np.asarray(col, np.int32).copy()
    N = wl.num_nodes
    rng = np.random.default_rng(7)
    bad = rng.choice(col.size, size=40, replace=False)
    col[bad[:20]] = -3
    col[bad[20:]] = N + 5
    v = 17  # pin 17's row ends before it starts
    off[v + 1] = off[v] - 1 if off[v] > 0 else off[v]
    off[N] = off[N] + 7  # the last node's row runs past nnz
    print(f"[case] walk table, corrupt graph W={walks} i64={offsets64}", flush=True)
    csr, tab = _both(off, col, wl.num_pins, wl.num_boards, walks, 3, 10, 11,
                     offsets64=offsets64)
    _assert_same(csr, tab, "corrupt graph")


def test_tiny_workload_matches_oracle(orc):
    wl = synth.WORKLOADS["tiny"]
    off, col, _ = synth.make_graph(wl)
    print("[case] walk table, tiny workload vs oracle", flush=True)
    csr, tab = _both(off, col, wl.num_pins, wl.num_boards, wl.walks, wl.hops, wl.T, wl.seed)
    ref = orc.build_neighborhoods(off, col, wl.num_pins, wl.seed, wl.walks, wl.hops, wl.T)
    _assert_same(tab, ref, "tiny vs oracle")
    _assert_same(csr, tab, "tiny")
