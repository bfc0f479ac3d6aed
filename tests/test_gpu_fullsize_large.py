"""GPU parity at full size, 10M pins + 2M boards (~56M edges), bf16, dims
1024 -> 2048 -> 512, 100 walks x 3 hops, T = 50, in the launch configuration
of the all-node job (inputs drawn on the GPU by synth.device_gen):

* the whole neighbourhood table -- ids, counts and fp32 weights of all 12M
  rows, and the total of edge steps -- bit-exact against the oracle, compared
  in six source ranges of 2M nodes;
* the embeddings of 128 targets (pins and boards spread over the id range,
  with the first and last node) through the oracle's Algorithm 2 with
  neighbourhoods walked on demand, for both layer dataflows.
The oracle's time limits the embedding targets (Algorithm 2 for 128 targets
projects about 330k layer-0 rows of 1024 -> 2048 in fp64).
"""

import gc

import numpy as np
import pytest
import torch

import synth
from helpers import check_embeddings, to_f64

pytestmark = pytest.mark.gpu

CHUNKS = 6


def _log(m):
    print(f"[gen] {m}", flush=True)


@pytest.fixture(scope="module")
def large():
    import paper_1806_01973_amd as ps
    from synth.device_gen import make_features_device, make_graph_device
    wl = synth.WORKLOADS["large"]
    print(f"[case] large: generating {wl.num_nodes} nodes on the GPU", flush=True)
    offsets, col, E = make_graph_device(wl, log=_log)
    x = make_features_device(wl, offsets, col, log=_log)
    gc.collect()
    torch.cuda.empty_cache()
    g = ps.DeviceGraph(offsets, col, wl.num_pins, wl.num_boards, offsets64=wl.offsets64)
    st = {"wl": wl, "g": g, "x": x, "E": E, "off_h": offsets.cpu().numpy(),
          "col_h": col.cpu().numpy(), "jobs": {}, "oracle_steps": 0, "checked": 0}
    yield st
    for job in st["jobs"].values():
        job.close()
    st.clear()
    gc.collect()
    torch.cuda.empty_cache()


def _job(st, dataflow):
    """The all-node job of one dataflow (the other one is released first)."""
    import paper_1806_01973_amd as ps
    if dataflow not in st["jobs"]:
        for k in list(st["jobs"]):
            st["jobs"].pop(k).close()
        st.pop("out", None)
        gc.collect()
        torch.cuda.empty_cache()
        wl = st["wl"]
        layers = [ps.DeviceLayer(L["Q"], L["q"], L["W"], L["w"], dtype=torch.bfloat16,
                                 dataflow=dataflow) for L in synth.make_layers(wl)]
        job = ps.EmbedAll(st["g"], layers, wl.walks, wl.hops, wl.T, wl.seed)
        st["out"] = job.run(st["x"])
        torch.cuda.synchronize()
        st["jobs"][dataflow] = job
        print(f"[case] large: embed_all {dataflow} done, steps={int(job.steps.item())}",
              flush=True)
    return st["jobs"][dataflow]


@pytest.mark.parametrize("chunk", range(CHUNKS))
def test_large_neighbourhood_table(orc, large, chunk):
    st = large
    wl = st["wl"]
    job = _job(st, "dense_then_pool")
    n = wl.num_nodes
    lo, hi = chunk * n // CHUNKS, (chunk + 1) * n // CHUNKS
    src = np.arange(lo, hi, dtype=np.int32)
    print(f"[case] large neighbourhoods, sources [{lo}, {hi})", flush=True)
    ridx, rcnt, rwts, steps = orc.build_neighborhoods(st["off_h"], st["col_h"], wl.num_pins,
                                                      wl.seed, wl.walks, wl.hops, wl.T,
                                                      sources=src)
    np.testing.assert_array_equal(job.nbr.idx[lo:hi].cpu().numpy(), ridx)
    np.testing.assert_array_equal(job.nbr.counts.view(torch.int16)[lo:hi].cpu().numpy()
                                  .view(np.uint16), rcnt)
    np.testing.assert_array_equal(job.nbr.weights[lo:hi].cpu().numpy().view(np.uint32),
                                  rwts.view(np.uint32))
    st["oracle_steps"] += int(steps)
    st["checked"] += hi - lo
    if st["checked"] == n:
        assert int(job.steps.item()) == st["oracle_steps"]
    print(f"[ok] large rows [{lo}, {hi}) bit-exact ({steps} edge steps)", flush=True)


@pytest.fixture(scope="module")
def large_reference(orc, large):
    st = large
    wl = st["wl"]
    rng = np.random.default_rng(3)
    targets = np.unique(np.concatenate([
        rng.choice(wl.num_pins, 96, replace=False),
        wl.num_pins + rng.choice(wl.num_boards, 30, replace=False),
        [0, wl.num_nodes - 1]])).astype(np.int32)
    print(f"[case] large: oracle Algorithm 2 for {len(targets)} targets", flush=True)
    smp = orc.minibatch_sample(targets, wl.K, st["off_h"], st["col_h"], wl.num_pins, wl.seed,
                               wl.walks, wl.hops, wl.T)
    s0 = smp["sets"][0]
    x_rows = to_f64(st["x"][torch.as_tensor(s0).long().cuda()])
    ref = orc.minibatch_embed_sampled(targets, s0, x_rows, smp, synth.make_layers(wl))
    print(f"[ok] large: |S| = {[len(s) for s in smp['sets']]}", flush=True)
    return targets, ref


@pytest.mark.parametrize("dataflow", ["dense_then_pool", "pool_then_dense"])
def test_large_embeddings(large, large_reference, dataflow):
    st = large
    targets, ref = large_reference
    _job(st, dataflow)
    got = to_f64(st["out"][torch.as_tensor(targets).long().cuda()])
    stats = check_embeddings(got, ref, st["wl"].dtype, f"large {dataflow}")
    print(f"[ok] large {dataflow}: {len(targets)} targets {stats}", flush=True)
