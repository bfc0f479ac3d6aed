"""GPU parity at full size for the two largest workloads, in the launch
configuration of the all-node job:

* large: 10M pins + 2M boards, bf16, dims 1024 -> 2048 -> 512, 100 walks x 3 hops
* shard: 80M pins + 20M boards (~1B CSR entries, int64 row offsets), bf16,
  dims 256 -> 512 -> 256, 50 walks x 3 hops, weights derived from counts

Inputs are drawn on the GPU (synth.device_gen). The oracle checks, one by one,
neighbourhood rows of 100k random sources (bit-exact) and the embeddings of 24
random nodes through Algorithm 2 with neighbourhoods walked on demand; the
embeddings of both layer dataflows (pool then dense, dense then pool) are
checked against the same oracle rows.
"""

import gc

import numpy as np
import pytest
import torch

import synth
from helpers import check_embeddings, to_f64
from synth.device_gen import make_features_device, make_graph_device

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name", ["large", "shard"])
def test_full_size_sampled(orc, name):
    import paper_1806_01973_amd as ps
    wl = synth.WORKLOADS[name]
    print(f"[case] full size {name}: generating {wl.num_nodes} nodes on the GPU", flush=True)
    log = lambda m: print(f"[gen] {m}", flush=True)
    offsets, col, E = make_graph_device(wl, log=log)
    x = make_features_device(wl, offsets, col, log=log)
    gc.collect()
    torch.cuda.empty_cache()
    g = ps.DeviceGraph(offsets, col, wl.num_pins, wl.num_boards, offsets64=wl.offsets64)
    off_h = offsets.cpu().numpy()
    col_h = col.cpu().numpy()
    rng = np.random.default_rng(5)
    src = np.sort(rng.choice(wl.num_nodes, 100_000, replace=False)).astype(np.int32)
    targets = np.concatenate([rng.choice(wl.num_pins, 16, replace=False),
                              wl.num_pins + rng.choice(wl.num_boards, 6, replace=False),
                              [0, wl.num_nodes - 1]]).astype(np.int32)
    ref = None
    for dataflow in ("pool_then_dense", "dense_then_pool"):
        print(f"[case] {name}: {E} edges; running embed_all {dataflow}", flush=True)
        layers = [ps.DeviceLayer(L["Q"], L["q"], L["W"], L["w"], dtype=torch.bfloat16,
                                 dataflow=dataflow) for L in synth.make_layers(wl)]
        job = ps.EmbedAll(g, layers, wl.walks, wl.hops, wl.T, wl.seed, weights=(name != "shard"))
        out = job.run(x)
        torch.cuda.synchronize()
        print(f"[case] {name}: embed_all done, steps={int(job.steps.item())}", flush=True)
        if ref is None:
            ridx, rcnt, rwts, _ = orc.build_neighborhoods(off_h, col_h, wl.num_pins, wl.seed,
                                                          wl.walks, wl.hops, wl.T, sources=src)
            sel = torch.as_tensor(src).long().cuda()
            np.testing.assert_array_equal(job.nbr.idx[sel].cpu().numpy(), ridx)
            np.testing.assert_array_equal(
                job.nbr.counts.view(torch.int16)[sel].cpu().numpy().view(np.uint16), rcnt)
            if job.nbr.weights is not None:
                np.testing.assert_array_equal(job.nbr.weights[sel].cpu().numpy().view(np.uint32),
                                              rwts.view(np.uint32))
            smp = orc.minibatch_sample(targets, wl.K, off_h, col_h, wl.num_pins, wl.seed,
                                       wl.walks, wl.hops, wl.T)
            s0 = smp["sets"][0]
            x_rows = to_f64(x[torch.as_tensor(s0).long().cuda()])
            ref = orc.minibatch_embed_sampled(targets, s0, x_rows, smp, synth.make_layers(wl))
            print(f"[ok] {name}: neighbourhoods match; |S| = {[len(s) for s in smp['sets']]}",
                  flush=True)
        got = to_f64(out[torch.as_tensor(targets).long().cuda()])
        stats = check_embeddings(got, ref, wl.dtype, f"{name} sampled {dataflow}")
        print(f"[ok] {name} {dataflow}: {stats}", flush=True)
        del job, out, layers
        gc.collect()
        torch.cuda.empty_cache()
    del x, g, offsets, col
    gc.collect()
    torch.cuda.empty_cache()
