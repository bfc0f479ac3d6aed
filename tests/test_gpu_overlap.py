"""GPU: the all-node job's schedule does not change its output.

With 262,144 to 4,194,304 pins the walks and the first layer's transform of a
leading share of the pins run beside each other on the CU-masked streams of a
caller-owned schedule, and the share follows the previous call's timing. The GEMMs sum every row in the same
order whatever the split, so every schedule must give the same bits as the
in-order one (walks, then the whole transform on the caller's stream):

* the 1.2M-node fp32 graph, both layer dataflows, side CU shares of 2/8, 3/8
  and 4/8, three calls in a row (the pin share moves between calls), the
  same graph in bf16, and a single layer (the overlapped layer is the last);
* a 4.5M-node bf16 graph with more pins than one 4,194,304-row chunk, whose
  first layer is chained and whose walk table fits in the first layer's output
  buffer, so it overlaps too (the walks reading that table), and a tiny graph
  (below the overlapped range: every share runs in order);
* int64 row offsets with weights derived from counts, at 2^18 pins (the
  smallest overlapped size) and 2^18 - 1 pins (in order);
* the overlapped call captured into a HIP graph and replayed.
The outputs themselves are checked against the oracle by the other GPU tests.
"""

import dataclasses

import pytest
import torch

import synth

pytestmark = pytest.mark.gpu


def _layers(wl, dtype, dataflow):
    import paper_1806_01973_amd as ps
    return [ps.DeviceLayer(L["Q"], L["q"], L["W"], L["w"], dtype=dtype, dataflow=dataflow)
            for L in synth.make_layers(wl)]


def _runs(g, layers, wl, x, shares, calls):
    import paper_1806_01973_amd as ps
    outs = []
    for k in shares:
        print(f"[case] share {k}/8", flush=True)
        job = ps.EmbedAll(g, layers, wl.walks, wl.hops, wl.T, wl.seed, overlap=k)
        for _ in range(calls if k else 1):
            out = job.run(x).clone()
            torch.cuda.synchronize()
            outs.append((k, out, job.nbr.idx.clone(), int(job.steps.item())))
        job.close()
    return outs


def _same(outs, what):
    k0, ref, ridx, rsteps = outs[0]
    assert k0 == 0
    for k, out, idx, steps in outs[1:]:
        assert steps == rsteps, f"{what} share {k}: steps"
        assert torch.equal(idx, ridx), f"{what} share {k}: neighbourhoods differ"
        assert torch.equal(out, ref), f"{what} share {k}: embeddings differ"


@pytest.fixture(scope="module")
def medium():
    import paper_1806_01973_amd as ps
    wl = synth.WORKLOADS["medium"]
    data = synth.make_workload(wl)
    g = ps.DeviceGraph(data["offsets"], data["col"], wl.num_pins, wl.num_boards)
    return wl, g, torch.as_tensor(data["x"]).cuda()


@pytest.mark.parametrize("dataflow", ["dense_then_pool", "pool_then_dense"])
def test_medium_schedules_agree(medium, dataflow):
    wl, g, x = medium
    print(f"[case] overlap schedules, 1.2M nodes f32 {dataflow}", flush=True)
    outs = _runs(g, _layers(wl, torch.float32, dataflow), wl, x, (0, 2, 3, 4), 3)
    _same(outs, f"medium {dataflow}")


def test_chunked_schedules_agree():
    import paper_1806_01973_amd as ps
    from synth.device_gen import make_features_device, make_graph_device
    base = synth.WORKLOADS["minibatch"]  # bf16, 256 -> 512 -> 256
    wl = dataclasses.replace(base.scaled(4_300_000, 200_000, "overlap-chunked"), walks=20)
    print("[case] schedules, 4.3M pins (chained first layer, overlapped) bf16", flush=True)
    offsets, col, _ = make_graph_device(wl)
    x = make_features_device(wl, offsets, col)
    g = ps.DeviceGraph(offsets, col, wl.num_pins, wl.num_boards)
    outs = _runs(g, _layers(wl, torch.bfloat16, "dense_then_pool"), wl, x, (0, 2), 2)
    _same(outs, "chunked")
    del outs, g, x, offsets, col
    torch.cuda.empty_cache()


def test_small_graph_and_bad_share():
    import paper_1806_01973_amd as ps
    wl = synth.WORKLOADS["tiny"]
    data = synth.make_workload(wl)
    g = ps.DeviceGraph(data["offsets"], data["col"], wl.num_pins, wl.num_boards)
    x = torch.as_tensor(data["x"]).cuda()
    print("[case] overlap below the pin threshold", flush=True)
    outs = _runs(g, _layers(wl, torch.float32, "dense_then_pool"), wl, x, (0, 7), 2)
    _same(outs, "tiny")
    for bad in (8, 0, -1):
        with pytest.raises(ps.PinsageError):
            ps.Schedule(bad)


def test_medium_graph_capture(medium):
    # The overlapped schedule forks and joins by events only, so the call can be
    # captured into a HIP graph on the caller's stream. Replays (with eager work
    # and synchronisations between them) must match the eager in-order result.
    import paper_1806_01973_amd as ps
    wl, g, x = medium
    layers = _layers(wl, torch.float32, "dense_then_pool")
    ref_job = ps.EmbedAll(g, layers, wl.walks, wl.hops, wl.T, wl.seed)
    ref = ref_job.run(x).clone()
    torch.cuda.synchronize()
    job = ps.EmbedAll(g, layers, wl.walks, wl.hops, wl.T, wl.seed, overlap=4)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    job.run(x, s)  # eager call first: times the split
    torch.cuda.synchronize()
    print("[case] overlap schedule captured into a graph, 1.2M nodes f32", flush=True)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=s):
        job.run(x, s)
    torch.cuda.synchronize()
    for rep in range(3):
        job.out.zero_()
        job.nbr.idx.fill_(-7)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        print(f"[case] replay {rep}", flush=True)
        assert torch.equal(job.nbr.idx, ref_job.nbr.idx), f"replay {rep}: neighbourhoods"
        assert torch.equal(job.out, ref), f"replay {rep}: embeddings"
        assert int(job.steps.item()) == int(ref_job.steps.item())
    del graph
    torch.cuda.synchronize()
    job.close()


def test_offsets64_count_weights_and_threshold():
    # int64 row offsets with weights derived from counts (no weight table), and
    # graphs at the pin-count threshold: 2^18 pins overlap, 2^18 - 1 do not.
    # Every schedule must match the in-order one bit for bit.
    import paper_1806_01973_amd as ps
    base = synth.WORKLOADS["medium"]
    for pins, boards, off64 in ((1 << 18, 60_000, True), ((1 << 18) - 1, 60_000, False)):
        wl = dataclasses.replace(base.scaled(pins, boards, "overlap-threshold"), walks=30)
        data = synth.make_workload(wl)
        g = ps.DeviceGraph(data["offsets"], data["col"], wl.num_pins, wl.num_boards,
                           offsets64=off64)
        x = torch.as_tensor(data["x"]).cuda()
        layers = _layers(wl, torch.float32, "dense_then_pool")
        print(f"[case] schedules, {pins} pins, offsets64={off64}, weights from counts",
              flush=True)
        outs = []
        for k in (0, 4, 4):
            job = ps.EmbedAll(g, layers, wl.walks, wl.hops, wl.T, wl.seed, weights=False,
                              overlap=k)
            out = job.run(x).clone()
            torch.cuda.synchronize()
            outs.append((k, out, job.nbr.idx.clone(), int(job.steps.item())))
            job.close()
        _same(outs, f"{pins} pins")


def test_medium_bf16_schedules_agree(medium):
    # bf16 storage: the first transform runs in the register-staged GEMM on the
    # side stream; the split must not change a bit either.
    wl, g, x = medium
    print("[case] overlap schedules, 1.2M nodes bf16 dense_then_pool", flush=True)
    layers = _layers(wl, torch.bfloat16, "dense_then_pool")
    outs = _runs(g, layers, wl, x.to(torch.bfloat16), (0, 4), 3)
    _same(outs, "medium bf16")


def test_medium_single_layer_schedules_agree(medium):
    # K = 1: the overlapped first layer is also the last one (its W GEMM writes
    # the output directly).
    wl, g, x = medium
    print("[case] overlap schedules, 1.2M nodes f32, one layer", flush=True)
    layers = _layers(wl, torch.float32, "dense_then_pool")[:1]
    outs = _runs(g, layers, wl, x, (0, 4), 2)
    _same(outs, "medium K=1")
