"""GPU: a graph carrying its walk table (pinsage_build_walk_table, set in
pinsage_graph_t.walk_table) gives every walk of the library the same bits as
the CSR walk (Sec. 3.2: the walk does not depend on the layout):

* neighbourhoods of all nodes and of a source list, on the tiny workload, a
  graph with out-of-range ids and malformed rows, and int64 row offsets;
* hard negatives (Sec. 3.3) on the on-chip path (walks x hops <= 16,384) and
  the global path, step totals included;
* the minibatch forward (Algorithm 2): frontier sets, embeddings and loss;
* the all-node job in order and overlapped (1.2M-node graph, the table the
  caller's instead of the job's own).
"""

import numpy as np
import pytest
import torch

import synth

pytestmark = pytest.mark.gpu


def _graph(off, col, P, B, offsets64=False):
    import paper_1806_01973_amd as ps
    return ps.DeviceGraph(off, col, P, B, offsets64=offsets64)


def _nb_same(a, b, what):
    (na, sa), (nb, sb) = a, b
    assert torch.equal(na.idx, nb.idx), f"{what}: idx"
    assert torch.equal(na.counts, nb.counts), f"{what}: counts"
    assert torch.equal(na.weights.view(torch.int32), nb.weights.view(torch.int32)), \
        f"{what}: weights"
    assert int(sa.item()) == int(sb.item()), f"{what}: steps"


def _corrupt_tiny():
    wl = synth.WORKLOADS["tiny"]
    off, col, _ = synth.make_graph(wl)
    off = np.asarray(off, np.int64).copy()
    col = np.asarray(col, np.int32).copy()
    N = wl.num_nodes
    rng = np.random.default_rng(5)
    bad = rng.choice(col.size, size=30, replace=False)
    col[bad[:15]] = -2
    col[bad[15:]] = N + 3
    off[23 + 1] = off[23] - 1 if off[23] > 0 else off[23]  # a row that ends before it starts
    return wl, off, col


@pytest.mark.parametrize("case", ["tiny", "corrupt", "int64"])
def test_neighborhoods(case):
    import paper_1806_01973_amd as ps
    wl = synth.WORKLOADS["tiny"]
    if case == "corrupt":
        wl, off, col = _corrupt_tiny()
    else:
        off, col, _ = synth.make_graph(wl)
    g = _graph(off, col, wl.num_pins, wl.num_boards, offsets64=case == "int64")
    print(f"[case] graph walk table, neighbourhoods {case}", flush=True)
    src = torch.as_tensor(np.random.default_rng(1).integers(0, wl.num_nodes, 777)
                          .astype(np.int32)).cuda()
    for walks in (40, 100):
        ref_all = ps.build_neighborhoods(g, walks, wl.hops, wl.T, wl.seed)
        ref_src = ps.build_neighborhoods(g, walks, wl.hops, wl.T, wl.seed, sources=src)
        g.build_walk_table()
        got_all = ps.build_neighborhoods(g, walks, wl.hops, wl.T, wl.seed)
        got_src = ps.build_neighborhoods(g, walks, wl.hops, wl.T, wl.seed, sources=src)
        torch.cuda.synchronize()
        g.drop_walk_table()
        _nb_same(ref_all, got_all, f"{case} all W={walks}")
        _nb_same(ref_src, got_src, f"{case} sources W={walks}")


@pytest.mark.parametrize("walks,hops,lo,hi", [(1024, 4, 100, 400), (4096, 4, 1999, 5000),
                                              (8192, 4, 1999, 5000)])
def test_hard_negatives(walks, hops, lo, hi):
    import paper_1806_01973_amd as ps
    wl = synth.WORKLOADS["medium"]
    off, col, _ = synth.make_graph(wl)
    g = _graph(off, col, wl.num_pins, wl.num_boards)
    q = torch.as_tensor(np.random.default_rng(3).integers(0, wl.num_pins, 300)
                        .astype(np.int32)).cuda()
    q[7] = -1  # an absent query
    print(f"[case] graph walk table, hard negatives {walks} x {hops}", flush=True)
    ref, rs = ps.hard_negatives(g, q, 6, 9, walks, hops, lo, hi, count_steps=True)
    g.build_walk_table()
    got, gs = ps.hard_negatives(g, q, 6, 9, walks, hops, lo, hi, count_steps=True)
    torch.cuda.synchronize()
    assert torch.equal(ref, got)
    assert int(rs.item()) == int(gs.item())


@pytest.mark.parametrize("hard_k", [0, 2])
def test_minibatch(hard_k):
    import paper_1806_01973_amd as ps
    wl = synth.WORKLOADS["tiny"]
    data = synth.make_workload(wl)
    g = _graph(data["offsets"], data["col"], wl.num_pins, wl.num_boards)
    layers = [ps.DeviceLayer(L["Q"], L["q"], L["W"], L["w"], dtype=torch.float32)
              for L in data["layers"]]
    x = torch.as_tensor(data["x"]).cuda()
    rng = np.random.default_rng(4)
    B, n_neg = 64, 50
    q, p, n = (torch.as_tensor(rng.integers(0, wl.num_pins, s).astype(np.int32)).cuda()
               for s in (B, B, n_neg))
    hard = (torch.as_tensor(rng.integers(-1, wl.num_pins, (B, hard_k)).astype(np.int32)).cuda()
            if hard_k else None)
    print(f"[case] graph walk table, minibatch hard_k={hard_k}", flush=True)
    mb = ps.Minibatch(g, layers, wl.walks, wl.hops, wl.T, wl.seed, B, n_neg, num_hard=hard_k)
    mb.run(x, q, p, n, 0.1, hard=hard)
    torch.cuda.synchronize()
    ref = (mb.loss.clone(), mb.z.clone(), mb.sizes(), int(mb.steps.item()))
    g.build_walk_table()
    mb.run(x, q, p, n, 0.1, hard=hard)
    torch.cuda.synchronize()
    assert mb.sizes() == ref[2]
    assert int(mb.steps.item()) == ref[3]
    assert torch.equal(mb.z, ref[1])
    assert torch.equal(mb.loss, ref[0])


@pytest.mark.parametrize("overlap", [0, 4])
def test_embed_all(overlap):
    import paper_1806_01973_amd as ps
    wl = synth.WORKLOADS["medium"]
    data = synth.make_workload(wl)
    g = _graph(data["offsets"], data["col"], wl.num_pins, wl.num_boards)
    layers = [ps.DeviceLayer(L["Q"], L["q"], L["W"], L["w"], dtype=torch.float32,
                             dataflow="dense_then_pool") for L in data["layers"]]
    x = torch.as_tensor(data["x"]).cuda()
    print(f"[case] graph walk table, embed_all overlap={overlap}", flush=True)
    job = ps.EmbedAll(g, layers, wl.walks, wl.hops, wl.T, wl.seed, overlap=overlap)
    job.run(x)
    torch.cuda.synchronize()
    ref = (job.out.clone(), job.nbr.idx.clone(), int(job.steps.item()))
    g.build_walk_table()
    for _ in range(2):
        job.run(x)
        torch.cuda.synchronize()
        assert int(job.steps.item()) == ref[2]
        assert torch.equal(job.nbr.idx, ref[1])
        assert torch.equal(job.out, ref[0])
    job.close()
