"""GPU parity: the MapReduce-inference variant of Sec. 3.4 (boards pool their
pins, pins their boards, featureless boards).

* Graph neighbourhoods bit for bit against the oracle (ids, multiplicities,
  fp32 weights) for every slot width (T up to 64, 128, 256), sampled and
  unsampled rows, the whole 1.2M-node graph (its huge boards sampled), int64
  row offsets, source subsets with invalid ids and NULL weights.
* The all-node job against the oracle: every row of the tiny graph (fp32 and
  bf16, both layer dataflows) and, on the 1.2M-node graph, a sample of pins
  and boards through the oracle's Algorithm 2 route on the same table.
"""

import dataclasses

import numpy as np
import pytest
import torch

import synth
from helpers import check_embeddings, to_f64, torch_dtype

pytestmark = pytest.mark.gpu


def _gpu_table(off, col, P, B, T, seed, sources=None, offsets64=None, weights=True):
    import paper_1806_01973_amd as ps
    g = ps.DeviceGraph(off, col, P, B, offsets64=offsets64)
    src = None if sources is None else torch.as_tensor(np.asarray(sources, np.int32)).cuda()
    nb = ps.build_graph_neighborhoods(g, T, seed, sources=src, weights=weights)
    torch.cuda.synchronize()
    return (nb.idx.cpu().numpy(), nb.counts.cpu().numpy(),
            None if nb.weights is None else nb.weights.cpu().numpy())


def _same(gpu, ref, what):
    np.testing.assert_array_equal(gpu[0], ref[0], err_msg=f"{what}: idx")
    np.testing.assert_array_equal(gpu[1], ref[1], err_msg=f"{what}: counts")
    if gpu[2] is not None:
        np.testing.assert_array_equal(gpu[2].view(np.uint32), ref[2].view(np.uint32),
                                      err_msg=f"{what}: weights")


@pytest.fixture(scope="module")
def tiny():
    wl = synth.WORKLOADS["tiny"]
    off, col, _ = synth.make_graph(wl)
    return wl, off, col


@pytest.mark.parametrize("T", [1, 8, 16, 37, 64, 100, 128, 200, 256])
def test_tiny_tables(orc, tiny, T):
    wl, off, col = tiny
    print(f"[case] graph neighbourhoods tiny T={T}", flush=True)
    gpu = _gpu_table(off, col, wl.num_pins, wl.num_boards, T, 11)
    _same(gpu, orc.graph_neighborhoods(off, col, 11, T), f"tiny T={T}")


def test_subsets_offsets64_no_weights(orc, tiny):
    wl, off, col = tiny
    src = np.array([2499, -3, 0, 2000, 77, 2500, 1999, 0], np.int32)
    print("[case] graph neighbourhoods subset / int64 offsets / NULL weights", flush=True)
    gpu = _gpu_table(off, col, wl.num_pins, wl.num_boards, 12, 4, sources=src, offsets64=True)
    _same(gpu, orc.graph_neighborhoods(off, col, 4, 12, sources=src), "subset")
    gi, gc, gw = _gpu_table(off, col, wl.num_pins, wl.num_boards, 12, 4, weights=False)
    ri, rc, _ = orc.graph_neighborhoods(off, col, 4, 12)
    assert gw is None
    np.testing.assert_array_equal(gi, ri)
    np.testing.assert_array_equal(gc, rc)


def test_invalid_entries_dropped(orc):
    # Node 0's row holds an id past the graph; it is dropped on both sides.
    off = np.array([0, 3, 4, 5, 6], np.int64)
    col = np.array([2, 99, 3, 0, 0, 0], np.int32)
    print("[case] graph neighbourhoods with an out-of-graph entry", flush=True)
    gpu = _gpu_table(off, col, 2, 2, 4, 1)
    _same(gpu, orc.graph_neighborhoods(off, col, 1, 4), "invalid entries")
    assert gpu[0][0, 0] == 2 and gpu[0][0, 1] == 3 and gpu[2][0, 0] == 0.5


def test_medium_table(orc):
    wl = synth.WORKLOADS["medium"]
    off, col, _ = synth.make_graph(wl)
    print("[case] graph neighbourhoods 1.2M nodes T=50", flush=True)
    gpu = _gpu_table(off, col, wl.num_pins, wl.num_boards, 50, wl.seed)
    _same(gpu, orc.graph_neighborhoods(off, col, wl.seed, 50), "medium")
    deg = np.diff(off)
    assert deg.max() > 50 and (gpu[1].sum(axis=1)[deg > 50] == 50).all()


def _layers(wl, dtype, dataflow):
    import paper_1806_01973_amd as ps
    data_layers = synth.make_layers(wl)
    return data_layers, [ps.DeviceLayer(L["Q"], L["q"], L["W"], L["w"], dtype=torch_dtype(dtype),
                                        dataflow=dataflow) for L in data_layers]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("dataflow", ["pool_then_dense", "dense_then_pool"])
def test_tiny_embedding(orc, tiny, dtype, dataflow):
    import paper_1806_01973_amd as ps
    wl, off, col = tiny
    wl = dataclasses.replace(wl, dtype=dtype)
    x = synth.make_features(wl, off, col)[: wl.num_pins]
    layers_np, layers = _layers(wl, dtype, dataflow)
    g = ps.DeviceGraph(off, col, wl.num_pins, wl.num_boards)
    job = ps.EmbedAllBipartite(g, layers, 20, 5)
    print(f"[case] bipartite embedding tiny {dtype} {dataflow}", flush=True)
    out = job.run(torch.as_tensor(x).to(device="cuda", dtype=torch_dtype(dtype)))
    torch.cuda.synchronize()
    idx, cnt, wts = orc.graph_neighborhoods(off, col, 5, 20)
    np.testing.assert_array_equal(job.nbr.idx.cpu().numpy(), idx)
    ref = orc.embed_all_bipartite(x, wl.num_nodes, layers_np, idx, wts)
    check_embeddings(to_f64(out), ref, dtype, f"bipartite tiny {dtype} {dataflow}")


def test_medium_embedding_sampled_rows(orc):
    import paper_1806_01973_amd as ps
    wl = synth.WORKLOADS["minibatch"]  # the 1.2M-node graph, bf16, 256/512/256
    off, col, _ = synth.make_graph(wl)
    x = synth.make_features(wl, off, col)[: wl.num_pins]
    layers_np, layers = _layers(wl, "bf16", "dense_then_pool")
    g = ps.DeviceGraph(off, col, wl.num_pins, wl.num_boards)
    job = ps.EmbedAllBipartite(g, layers, 50, wl.seed)
    print("[case] bipartite embedding 1.2M nodes bf16, sampled rows", flush=True)
    out = job.run(torch.as_tensor(x).to(device="cuda", dtype=torch.bfloat16))
    torch.cuda.synchronize()
    idx, cnt, wts = orc.graph_neighborhoods(off, col, wl.seed, 50)
    np.testing.assert_array_equal(job.nbr.idx.cpu().numpy(), idx)
    rng = np.random.default_rng(6)
    rows = np.concatenate([rng.choice(wl.num_pins, 300, replace=False),
                           wl.num_pins + rng.choice(wl.num_boards, 100, replace=False)])
    x_all = np.zeros((wl.num_nodes, wl.d_in), np.float64)
    x_all[: wl.num_pins] = x
    ref = orc.minibatch_embed(rows.astype(np.int32), x_all, layers_np, idx, wts)
    got = out[torch.as_tensor(rows).long().cuda()]
    check_embeddings(to_f64(got), ref, "bf16", "bipartite medium sampled")
