"""Benchmark: the PinSage hot path on one MI355X.

Default (the headline line): all-node embedding of the largest single-GPU
shard: 80M pins + 20M boards (~0.49B undirected edges, int64 row offsets),
features 256-d bf16, dims 256 -> 512 -> 256 with fp32 accumulation, 50 walks x
3 hops, T = 50. One step = importance neighbourhoods of every node, then K = 2
CONVOLVE layers over every node, layer by layer (Sec. 3.4). Inputs are drawn
on the device and resident in HBM before timing starts. The layers run in the
dense-then-pool order (the neighbour half of W applied per pin before the
weighted mean, which is linear); the printed order of Algorithm 1 needs the
82 GB table P and is parity-tested, not timed, at this size.

Other workloads (measurement of the other rows; not the headline):
  --workload tiny | medium | large  all-node embedding of that graph (medium:
                                    1M pins + 200k boards, fp32, where the
                                    first transform runs beside the walks on
                                    CU-masked streams, `--overlap`)
  --workload minibatch              one step = the minibatch forward of
                                    Algorithm 2 (2,048 pairs, 500 shared
                                    negatives) plus the loss of Eq. 1
  --workload minibatch --hard-neg K  the same step preceded by mining K hard
                                    negatives per query (Sec. 3.3), which join
                                    every pair's negatives in the loss
  --workload bipartite              one step = the MapReduce-inference variant
                                    of Sec. 3.4 on the 1.2M-node graph: graph
                                    neighbourhoods (T = 50, long rows sampled),
                                    2 layers over all nodes, featureless boards
  --workload hardneg                one step = hard negative items (Sec. 3.3)
                                    for 2,048 query pins of the 1.2M-node
                                    graph: 32768 walks x 4 landings each
                                    (--hn-walks, --hn-hops; budgets up to
                                    16,384 landings count visits in LDS,
                                    larger ones buffer the landings and count
                                    them by hash partition), ranks 2000-5000,
                                    --hard-neg draws per query

Prints one JSON line: throughput of the whole step, walk steps/s, per-kernel
times from hipEvents recorded around every launch in the timed region, the
roofline of the dominant kernel and the CPU oracle timed on a bounded sample
of the same workload.

  python bench.py [--steps K] [--warmup W] [--workload shard] [--no-cpu-baseline]
  python bench.py --copy-calibration   # plain copy of a known size, for counter scaling
  python bench.py --layer 1024,2048,512 --rows 4000000 --dtype bf16   # one layer, for counters
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "node embeddings/sec (K=2 layerwise, all nodes) + walk steps/sec, 1 MI355X"
HBM_PEAK_GBS = 8000.0
MFMA_PEAK_TFLOPS = {"f32": 157.3, "bf16": 2500.0}
PROFILE_DIR = os.path.join(ROOT, "profiles")
DEFAULT_STEPS = {"tiny": 20, "medium": 20, "minibatch": 20, "large": 4, "shard": 5, "hardneg": 20,
                 "bipartite": 20}
DEFAULT_WARMUP = {"tiny": 3, "medium": 3, "minibatch": 3, "large": 1, "shard": 1, "hardneg": 3,
                  "bipartite": 3}
# Hard negative workload: queries per step, walks and landings per query, the
# rank window [lo, hi) (ranks 2000-5000 counted from 1). At 32,768 x 4
# landings the window is decided by visit counts (at 4,096 x 4, the LDS
# kernel's budget, it falls among pins visited once).
HN_QUERIES, HN_WALKS, HN_HOPS, HN_LO, HN_HI = 2048, 32768, 4, 1999, 5000
# Hard negatives mined inside the minibatch step (--hard-neg): walks per pair.
MB_HN_WALKS = 4096
DEVICE_GENERATED = ("large", "shard")


def log(msg: str) -> None:
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def kernel_source_hash(name: str) -> str:
    """Hash of a kernel source file and the local device headers it includes
    (kernels.h, the host-side launch declarations, is left out)."""
    csrc = os.path.join(ROOT, "paper_1806_01973_amd", "csrc")
    h = hashlib.sha256()
    with open(os.path.join(csrc, name), "rb") as f:
        text = f.read()
    h.update(text)
    for line in text.decode().splitlines():
        line = line.strip()
        if line.startswith('#include "') and line.split('"')[1] != "kernels.h":
            inc = os.path.join(csrc, line.split('"')[1])
            if os.path.exists(inc):
                with open(inc, "rb") as f:
                    h.update(f.read())
    return h.hexdigest()[:16]


def load_traffic(kernel_file: str, workload: str):
    """Measured HBM bytes per launch of a kernel, if a counter summary exists for
    the current source of that kernel (else None)."""
    path = os.path.join(PROFILE_DIR, "traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        table = json.load(f)
    ent = table.get(f"{kernel_file}:{workload}")
    if not ent or ent.get("source_sha") != kernel_source_hash(kernel_file):
        return None
    return ent


def copy_calibration(gib: float = 1.0, reps: int = 5) -> None:
    import torch
    n = int(gib * (1 << 30)) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes": n * 4, "reps": reps}), flush=True)


def host_cpu() -> dict:
    """The host CPU the oracle ran on: model, logical CPUs, physical cores."""
    model, phys = None, set()
    try:
        with open("/proc/cpuinfo") as f:
            pid = core = None
            for line in f:
                key, _, val = line.partition(":")
                key, val = key.strip(), val.strip()
                if key == "model name" and model is None:
                    model = val
                elif key == "physical id":
                    pid = val
                elif key == "core id":
                    core = val
                elif not key and pid is not None and core is not None:
                    phys.add((pid, core))
                    pid = core = None
            if pid is not None and core is not None:
                phys.add((pid, core))
    except OSError:
        pass
    return {"model": model, "logical_cpus": os.cpu_count(), "physical_cores": len(phys) or None}


def random_read_calibration(table_gib: int = 16, steps: int = 32, reps: int = 3) -> None:
    """Dependent random reads per second (the library's calibration kernel):
    4-, 8- and 16-byte elements from a table_gib table, and 16-byte elements
    from its first 256 MiB, at several numbers of chains in flight."""
    import torch
    from paper_1806_01973_amd import _lib
    L = _lib.lib()
    table = torch.empty(table_gib << 30, dtype=torch.uint8, device="cuda")  # never written
    chains_max = 16384 * 256
    sink = torch.empty(chains_max, dtype=torch.int32, device="cuda")
    stream = torch.cuda.current_stream()
    out = {"table_bytes": table.numel(), "steps": steps, "reps": reps}
    for name, nbytes, eb in (("4B", table.numel(), 4), ("8B", table.numel(), 8),
                             ("16B", table.numel(), 16), ("16B_256MiB", 256 << 20, 16)):
        for chains in (2048 * 256, 8192 * 256, chains_max):
            def launch():
                _lib.check(L.pinsage_profile_random_reads(table.data_ptr(), nbytes, eb, steps,
                                                          sink.data_ptr(), chains,
                                                          stream.cuda_stream), "random reads")
            launch()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for _ in range(reps):
                launch()
            e1.record(stream)
            torch.cuda.synchronize()
            ms = e0.elapsed_time(e1) / reps
            out[f"reads_per_s_{name}_chains{chains}"] = chains * steps / (ms * 1e-3)
    print(json.dumps(out), flush=True)


def random_gather_calibration(targets: int = 8_000_000, reps: int = 3) -> None:
    """Random row gathers per second in the importance pool's access pattern
    (the library's calibration kernel): 512-byte rows from tables of 1, 4 and
    16 GiB and from one the size of the 100M-node shard's R table (80M rows),
    50 rows per target, and 1 KB rows from a table of the same size, 32 rows per
    target."""
    import torch
    from paper_1806_01973_amd import _lib
    L = _lib.lib()
    shard_r = 80_000_000 * 512
    table = torch.empty(shard_r, dtype=torch.uint8, device="cuda")  # never written
    sink = torch.zeros(1, dtype=torch.int32, device="cuda")
    stream = torch.cuda.current_stream()
    out = {"targets": targets, "reps": reps}
    for name, nbytes, rb, per in (("512B_1GiB", 1 << 30, 512, 50), ("512B_4GiB", 4 << 30, 512, 50),
                                  ("512B_16GiB", 16 << 30, 512, 50),
                                  ("512B_shardR", shard_r, 512, 50), ("1KB_shardR", shard_r, 1024, 32)):
        def launch():
            _lib.check(L.pinsage_profile_random_gathers(table.data_ptr(), nbytes, rb, targets, per,
                                                        1, sink.data_ptr(), stream.cuda_stream),
                       "random gathers")
        launch()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(reps):
            launch()
        e1.record(stream)
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / reps
        out[f"gather_GBs_{name}"] = targets * per * rb / (ms * 1e-3) / 1e9
        out[f"ms_{name}"] = ms
    print(json.dumps(out), flush=True)


def load_inputs(wl, dataflow="pool_then_dense", pool="importance"):
    """Inputs on the GPU plus host views the CPU baseline needs."""
    import numpy as np
    import torch

    import paper_1806_01973_amd as ps
    import synth

    tdt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    t0 = time.perf_counter()
    if wl.name in DEVICE_GENERATED:
        from synth.device_gen import make_features_device, make_graph_device
        offsets, col, E = make_graph_device(wl, log=log)
        x = make_features_device(wl, offsets, col, log=log)
        host = {"offsets": offsets.cpu().numpy(), "col": col.cpu().numpy()}
        x_rows = lambda n: x[:n].float().cpu().numpy()
    else:
        data = synth.make_workload(wl)
        offsets, col, E = data["offsets"], data["col"], data["num_edges"]
        x = torch.as_tensor(data["x"]).to(device="cuda", dtype=tdt)
        host = {"offsets": offsets, "col": col}
        x_rows = lambda n: data["x"][:n]
    layers_np = synth.make_layers(wl)
    g = ps.DeviceGraph(offsets, col, wl.num_pins, wl.num_boards, offsets64=wl.offsets64)
    layers = [ps.DeviceLayer(L["Q"], L["q"], L["W"], L["w"], dtype=tdt, dataflow=dataflow,
                             pool=pool) for L in layers_np]
    torch.cuda.synchronize()
    log(f"inputs for {wl.name}: {wl.num_nodes} nodes, {E} edges in "
        f"{time.perf_counter() - t0:.1f}s")
    return {"g": g, "x": x, "layers": layers, "layers_np": layers_np, "num_edges": int(E),
            "host": host, "x_rows": x_rows}


def cpu_baseline_embed(inp, wl, threads: int) -> dict:
    """The oracle as it stands, on a bounded sample of the same workload:
    neighbourhoods of a node sample, and each layer on a row sample (pins
    projected in the same pin:node proportion). Extrapolated per node."""
    import numpy as np
    import oracle

    N, P = wl.num_nodes, wl.num_pins
    n_walk = min(N, 1_500_000)
    p = P / N
    flops_row = 0.0
    d_prev = wl.d_in
    for _ in range(wl.K):
        flops_row += 2 * (p * d_prev * wl.m + (d_prev + wl.m) * wl.d_out)
        d_prev = wl.d_out
    n_rows = int(min(N, 400_000, 600e9 / flops_row))
    rng = np.random.default_rng(123)
    src = np.sort(rng.choice(N, n_walk, replace=False)).astype(np.int32)
    t0 = time.perf_counter()
    idx, cnt, wts, steps = oracle.build_neighborhoods(inp["host"]["offsets"], inp["host"]["col"],
                                                      P, wl.seed, wl.walks, wl.hops, wl.T,
                                                      sources=src, nthreads=threads)
    t_walk = time.perf_counter() - t0
    # Layer sample: rows [0, n_rows) of the node features, n_transform pins
    # among them, neighbour ids folded into that range.
    n_tr = max(1, int(round(n_rows * p)))
    idx_s = np.where(idx[:n_rows] >= 0, idx[:n_rows] % n_tr, -1).astype(np.int32)
    wts_s = wts[:n_rows]
    h = inp["x_rows"](n_rows)
    t_layers = 0.0
    for L in inp["layers_np"]:
        t0 = time.perf_counter()
        h = oracle.convolve_layer(h, n_tr, L["Q"], L["q"], L["W"], L["w"], idx_s, wts_s,
                                  nthreads=threads)
        t_layers += time.perf_counter() - t0
    per_node = t_walk / n_walk + t_layers / n_rows
    return {"value": 1.0 / per_node, "unit": "node embeddings/s", "cores": threads,
            "kind": "oracle",
            "sample": (f"neighbourhoods of {n_walk} random nodes ({t_walk:.1f}s, "
                       f"{steps / t_walk:.3g} walk steps/s) + all {wl.K} layers on {n_rows} "
                       f"rows with {n_tr} projected pins ({t_layers:.1f}s), fp64, extrapolated "
                       f"per node"),
            "walk_steps_per_s": steps / t_walk}


def kernel_table(prof, steps):
    kernels = {}
    for name, (n_launch, ms) in prof.items():
        if n_launch:
            kernels[name] = {"launches": n_launch, "avg_ms": ms / n_launch,
                             "ms_per_step": ms / steps}
    return kernels


def chained_layer(L) -> bool:
    """Layers whose Q transform and neighbour half of W run as one chained
    kernel in the library (dense then pool, bf16, d_in = d_out = 256, m a
    multiple of 32 up to 2048); their work is timed as gemm_qr."""
    import torch
    return (L.dataflow == "dense_then_pool" and getattr(L, "dtype", None) == torch.bfloat16
            and L.d_in == 256
            and L.d_out == 256 and L.m % 32 == 0 and 0 < L.m <= 2048)


def fused_layer(L, T) -> bool:
    """Layers whose pool and W run as one kernel in the library (dense then
    pool, bf16, d_in = d_out = 256, T <= 64); timed as pool_w."""
    import torch
    return (L.dataflow == "dense_then_pool" and getattr(L, "dtype", None) == torch.bfloat16
            and L.d_in == 256 and L.d_out == 256 and 1 <= T <= 64)


def add_rooflines(kernels, wl, layers, N, n_transform, live_entries, weights_stored,
                  walk_steps, steps):
    """Algorithmic work per launch and achieved rates. A step's work of a kernel
    class is divided by its launches per step (large layers run in row chunks)."""
    esz = 2 if wl.dtype == "bf16" else 4
    peak_tf = MFMA_PEAK_TFLOPS[wl.dtype]
    idx_bytes = N * wl.T * 4 + (N * wl.T * 4 if weights_stored else N * wl.T * 2)

    def per_launch(name, per_step):
        return per_step / (kernels[name]["launches"] / steps)

    # The pool gathers m-wide rows of P (pool then dense) or d_out-wide rows of
    # R = P W_n^T (dense then pool); the W GEMM then has K = d_in + m, resp. d_in.
    split = [L.dataflow == "dense_then_pool" for L in layers]
    width = [L.d_out if sp else L.m for L, sp in zip(layers, split)]
    fused = [fused_layer(L, wl.T) for L in layers]
    if "pool" in kernels:
        k = kernels["pool"]
        k["algo_bytes_per_launch"] = per_launch(
            "pool", sum(live_entries * w * esz + idx_bytes + N * w * esz
                        for w, fu in zip(width, fused) if not fu))
        k["achieved_GBs"] = k["algo_bytes_per_launch"] / (k["avg_ms"] * 1e-3) / 1e9
        k["frac_hbm"] = k["achieved_GBs"] / HBM_PEAK_GBS
    if "pool_w" in kernels:
        # Gathered rows, the neighbourhood table, the self rows and the output;
        # the W_s product's flops beside them.
        k = kernels["pool_w"]
        k["algo_bytes_per_launch"] = per_launch(
            "pool_w", sum(live_entries * L.d_out * esz + idx_bytes + N * L.d_in * esz
                          + N * L.d_out * esz for L, fu in zip(layers, fused) if fu))
        k["achieved_GBs"] = k["algo_bytes_per_launch"] / (k["avg_ms"] * 1e-3) / 1e9
        k["frac_hbm"] = k["achieved_GBs"] / HBM_PEAK_GBS
        k["algo_flops_per_launch"] = per_launch(
            "pool_w", sum(2.0 * N * L.d_in * L.d_out for L, fu in zip(layers, fused) if fu))
        k["achieved_TFLOPs"] = k["algo_flops_per_launch"] / (k["avg_ms"] * 1e-3) / 1e12
    chained = [chained_layer(L) for L in layers]
    for name, fl in (("gemm_q", sum(2.0 * n_transform * L.d_in * L.m
                                    for L, ch in zip(layers, chained) if not ch)),
                     ("gemm_r", sum(2.0 * n_transform * L.m * L.d_out
                                    for L, sp, ch in zip(layers, split, chained) if sp and not ch)),
                     ("gemm_qr", sum(2.0 * n_transform * (L.d_in * L.m + L.m * L.d_out)
                                     for L, ch in zip(layers, chained) if ch)),
                     ("gemm_w", sum(2.0 * N * (L.d_in + (0 if sp else L.m)) * L.d_out
                                    for L, sp, fu in zip(layers, split, fused) if not fu))):
        if name in kernels:
            k = kernels[name]
            k["algo_flops_per_launch"] = per_launch(name, fl)
            k["achieved_TFLOPs"] = k["algo_flops_per_launch"] / (k["avg_ms"] * 1e-3) / 1e12
            k["frac_mfma"] = k["achieved_TFLOPs"] / peak_tf
    if "walk_topt" in kernels and walk_steps:
        walk_rates(kernels["walk_topt"], per_launch("walk_topt", walk_steps), wl.offsets64,
                   table=kernels.get("walk_table", {}).get("launches", 0) > 0)


# Each edge step of a walk reading the CSR takes the offset pair of its node and
# one neighbour id at unrelated addresses; with the walk table, one 16-byte
# entry. A random read moves a 64-byte sector at most.
WALK_SECTOR_BYTES = 64
# Dependent random reads per second served from a 16 GiB table, 16-byte
# elements, 0.5-4M chains in flight (pinsage_profile_random_reads, the
# --random-read-calibration mode; 61.9-63.4 G/s on two boxes, see
# profiles/random_read_calibration.md). Every edge step needs at least one such
# read (the neighbour at a uniform position of the node's row), so this rate,
# not HBM bytes, bounds the walks.
RANDOM_READS_PER_S = 62.5e9


def walk_rates(k, edge_steps_per_launch, offsets64, table=False):
    """Rates of a walk kernel: algorithmic bytes per edge step (the offset pair
    and a column id, or one 16-byte walk-table entry) against the HBM peak;
    the time the step's random reads would take as whole 64-byte sectors at
    that peak (transaction floor); and the time one dependent random read per
    step takes at the chip's measured random-read rate (random-read floor)."""
    off_b = 8 if offsets64 else 4
    step_bytes = 16 if table else 2 * off_b + 4
    reads_per_step = 1 if table else 2
    k["walk_table"] = bool(table)
    k["edge_steps_per_launch"] = edge_steps_per_launch
    k["algo_bytes_per_launch"] = edge_steps_per_launch * step_bytes
    k["achieved_GBs"] = k["algo_bytes_per_launch"] / (k["avg_ms"] * 1e-3) / 1e9
    k["frac_hbm"] = k["achieved_GBs"] / HBM_PEAK_GBS
    k["edge_steps_per_s"] = edge_steps_per_launch / (k["avg_ms"] * 1e-3)
    floor_ms = (edge_steps_per_launch * reads_per_step * WALK_SECTOR_BYTES
                / (HBM_PEAK_GBS * 1e9) * 1e3)
    k["transaction_floor_ms"] = floor_ms
    k["frac_of_transaction_floor"] = floor_ms / k["avg_ms"]
    rr_ms = edge_steps_per_launch / RANDOM_READS_PER_S * 1e3
    k["random_read_floor_ms"] = rr_ms
    k["frac_of_random_read_floor"] = rr_ms / k["avg_ms"]


def roofline_of(kernels, wl):
    dominant = max(kernels, key=lambda n: kernels[n]["ms_per_step"])
    kd = kernels[dominant]
    if dominant in ("gemm_q", "gemm_r", "gemm_w", "gemm_qr"):
        return {"kernel": dominant, "bound": "mfma", "achieved": kd["achieved_TFLOPs"],
                "peak": MFMA_PEAK_TFLOPS[wl.dtype], "unit": "TFLOP/s", "frac": kd["frac_mfma"],
                "traffic": None}
    src_file = {"pool": "pool.hip", "pool_w": "poolw.hip", "walk_topt": "walk.hip",
                "hard_neg": "hardneg.hip"}.get(dominant, "")
    tr = load_traffic(src_file, wl.name) if src_file else None
    frac = (kd["achieved_GBs"] / HBM_PEAK_GBS) if "achieved_GBs" in kd else None
    walk_like = "edge_steps_per_launch" in kd
    out = {"kernel": dominant, "bound": "hbm", "achieved": kd.get("achieved_GBs"),
           "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": frac,
           "traffic": None if tr is None else tr["bytes_per_launch"],
           "bytes": ("algorithmic (the edge steps' reads: one 16-byte walk-table entry, or "
                     "an offset pair and a column id, per step)" if walk_like else
                     "algorithmic (every gathered row counted once per use)")}
    if walk_like:
        # Walk kernels are bound by the rate of dependent random reads, not by
        # HBM bytes: their time against that floor sits beside the HBM figures.
        out["random_read_floor_ms"] = kd.get("random_read_floor_ms")
        out["frac_of_random_read_floor"] = kd.get("frac_of_random_read_floor")
    if frac is not None and frac > 1.0:
        # More algorithmic bytes per second than HBM can deliver: the caches
        # (L2, MALL) serve part of the re-gathered rows, so this is not an HBM
        # fraction.
        out["cache_resident"] = True
    if tr is not None:
        out["traffic_GBs"] = tr["bytes_per_launch"] / (kd["avg_ms"] * 1e-3) / 1e9
        out["traffic_frac"] = out["traffic_GBs"] / HBM_PEAK_GBS
        out["traffic_profile"] = tr.get("profile")
    return out


STEP_MS: list = []  # per-step times of the headline's timed region (ms)


def timed(run, steps, warmup, stream=None):
    """Runs `warmup` untimed steps, then times exactly `steps` steps between two
    device synchronisations. Per-step durations are also taken with events on
    the step's stream (STEP_MS), for the median."""
    import torch

    import paper_1806_01973_amd as ps
    for i in range(warmup):
        run(i)
    torch.cuda.synchronize()
    log(f"warmup done ({warmup} steps)")
    st = stream if stream is not None else torch.cuda.current_stream()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    ps.profile_enable(True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev[0].record(st)
    for i in range(steps):
        run(warmup + i)
        ev[i + 1].record(st)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    prof = ps.profile_read()
    ps.profile_enable(False)
    STEP_MS[:] = [ev[i].elapsed_time(ev[i + 1]) for i in range(steps)]
    log(f"timed {steps} steps in {elapsed:.3f}s")
    return elapsed, prof


def bench_embed_all(args, wl, inp):
    import torch

    import paper_1806_01973_amd as ps
    # Graphs of 2^18 to 2^22 pins run the walks beside the first transform.
    # Larger ones run in order: their walks are bound by dependent random reads
    # and slow down beside the transform by about as much as it would save
    # (the library would overlap the shard's chained first layer, but at
    # 2/8 of the CUs that measured 1345 ms per step against 1341-1351 in order
    # on the same box, within the spread of runs).
    overlapped = bool(args.overlap) and (1 << 18) <= wl.num_pins <= (1 << 22)
    job = ps.EmbedAll(inp["g"], inp["layers"], wl.walks, wl.hops, wl.T, wl.seed,
                      weights=wl.name != "shard", overlap=args.overlap if overlapped else 0)
    # A stream of its own: the library's side streams then overlap freely with
    # it (the legacy default stream would wait for them at every launch).
    stream = torch.cuda.Stream()
    stream.wait_stream(torch.cuda.current_stream())
    mlp = inp.get("mlp")
    if mlp is not None:
        z = torch.empty((wl.num_nodes, mlp.d_out), dtype=mlp.dtype, device="cuda")
        mws = torch.empty(max(1, mlp_workspace(mlp, wl.num_nodes)), dtype=torch.uint8,
                          device="cuda")

    def step(i):
        h = job.run(inp["x"], stream)
        if mlp is not None:
            ps.output_mlp(mlp, h, out=z, workspace=mws, stream=stream)

    elapsed, prof = timed(step, args.steps, args.warmup, stream)
    N = wl.num_nodes
    walk_steps = int(job.steps.item())
    kernels = kernel_table(prof, args.steps)
    live = sum(int((job.nbr.idx[r0:r0 + (1 << 22)] >= 0).sum(dtype=torch.int64).item())
               for r0 in range(0, N, 1 << 22))
    add_rooflines(kernels, wl, inp["layers"], N, wl.num_pins, live, job.nbr.weights is not None,
                  walk_steps, args.steps)
    value = N * args.steps / elapsed
    layer_ms = sum(v["ms_per_step"] for k, v in kernels.items()
                   if k in ("gemm_q", "gemm_r", "gemm_qr", "pool", "pool_w", "gemm_w"))
    extra = {"walk_steps_per_s": kernels.get("walk_topt", {}).get("edge_steps_per_s"),
             # N over the layer kernels' time alone (walks excluded), hipEvents;
             # only in the in-order schedule (overlapped launches share the chip).
             "layers_embeddings_per_s": (N / (layer_ms * 1e-3)
                                         if layer_ms and not overlapped else None),
             "config_extra": {"nodes": N, "walk_steps_per_step": walk_steps,
                              # first layer's transform beside the walks on this
                              # many eighths of the CUs (0: in order); its launches
                              # and the walk's then time their shared duration
                              "overlap_cu_eighths": args.overlap if overlapped else 0}}
    if overlapped:
        # The walk kernel alone on every CU (outside the timed steps), next to
        # its rate on its share of the CUs inside the overlapped step.
        ps.profile_enable(True)
        for _ in range(3):
            ps.build_neighborhoods(inp["g"], wl.walks, wl.hops, wl.T, wl.seed, out=job.nbr,
                                   count_steps=False, stream=stream)
        torch.cuda.synchronize()
        n_w, ms_w = ps.profile_read()["walk_topt"]
        ps.profile_enable(False)
        extra["walk_steps_per_s_all_cus"] = walk_steps / (ms_w / n_w * 1e-3)
    if compare_dataflow(args, wl):
        # The other evaluation order of the same layers, timed the same way
        # (same inputs, same steps), for comparison only.
        other = "pool_then_dense" if args.dataflow == "dense_then_pool" else "dense_then_pool"
        alt_layers = [ps.DeviceLayer(L.Q, L.q, L.W, L.w, dtype=L.dtype, dataflow=other,
                                     pool=L.pool) for L in inp["layers"]]
        job.close()
        del job
        torch.cuda.empty_cache()
        alt = ps.EmbedAll(inp["g"], alt_layers, wl.walks, wl.hops, wl.T, wl.seed,
                          weights=wl.name != "shard", overlap=args.overlap if overlapped else 0)
        main_steps = list(STEP_MS)  # the headline's per-step times, kept
        alt_elapsed, _ = timed(lambda i: alt.run(inp["x"], stream), args.steps, args.warmup)
        STEP_MS[:] = main_steps
        extra["alt_dataflow"] = {"dataflow": other, "value": N * args.steps / alt_elapsed,
                                 "ms_per_step": 1e3 * alt_elapsed / args.steps}
        alt.close()
    else:
        job.close()
    return value, "node embeddings/s", METRIC, elapsed, kernels, extra


def bench_bipartite(args, wl, inp):
    """The MapReduce-inference variant of Sec. 3.4 on the same graph and layers:
    graph neighbourhoods (T per node, long rows sampled), then the layers over
    every node with featureless boards (x holds the pins' rows only)."""
    import torch

    import paper_1806_01973_amd as ps
    job = ps.EmbedAllBipartite(inp["g"], inp["layers"], wl.T, wl.seed)
    x_pins = inp["x"][: wl.num_pins]
    stream = torch.cuda.current_stream()
    elapsed, prof = timed(lambda i: job.run(x_pins, stream), args.steps, args.warmup)
    N = wl.num_nodes
    kernels = kernel_table(prof, args.steps)
    live = sum(int((job.nbr.idx[r0:r0 + (1 << 22)] >= 0).sum(dtype=torch.int64).item())
               for r0 in range(0, N, 1 << 22))
    add_rooflines(kernels, wl, inp["layers"], N, N, live, True, 0, args.steps)
    value = N * args.steps / elapsed
    extra = {"walk_steps_per_s": None,
             "config_extra": {"nodes": N, "neighbourhood_entries": live}}
    metric = ("node embeddings/sec (K=2 layerwise, all nodes), MapReduce inference variant "
              "(Sec. 3.4: graph neighbourhoods, featureless boards), 1 MI355X")
    return value, "node embeddings/s", metric, elapsed, kernels, extra


def cpu_baseline_bipartite(inp, wl, threads: int) -> dict:
    """The oracle on a bounded sample of the variant: graph neighbourhoods of
    every node, and each layer on a row sample with every sampled row
    projected. Extrapolated per node."""
    import numpy as np
    import oracle

    N = wl.num_nodes
    t0 = time.perf_counter()
    idx, cnt, wts = oracle.graph_neighborhoods(inp["host"]["offsets"], inp["host"]["col"],
                                               wl.seed, wl.T, nthreads=threads)
    t_nbr = time.perf_counter() - t0
    flops_row = 0.0
    d_prev = wl.d_in
    for _ in range(wl.K):
        flops_row += 2 * (d_prev * wl.m + (d_prev + wl.m) * wl.d_out)
        d_prev = wl.d_out
    n_rows = int(min(N, 400_000, 600e9 / flops_row))
    idx_s = np.where(idx[:n_rows] >= 0, idx[:n_rows] % n_rows, -1).astype(np.int32)
    h = inp["x_rows"](n_rows)
    t_layers = 0.0
    for L in inp["layers_np"]:
        t0 = time.perf_counter()
        h = oracle.convolve_layer(h, n_rows, L["Q"], L["q"], L["W"], L["w"], idx_s, wts[:n_rows],
                                  nthreads=threads)
        t_layers += time.perf_counter() - t0
    per_node = t_nbr / N + t_layers / n_rows
    return {"value": 1.0 / per_node, "unit": "node embeddings/s", "cores": threads,
            "kind": "oracle",
            "sample": (f"graph neighbourhoods of all {N} nodes ({t_nbr:.1f}s) + all {wl.K} "
                       f"layers on {n_rows} rows, every row projected ({t_layers:.1f}s), fp64, "
                       f"extrapolated per node")}


def mlp_workspace(mlp, n):
    import ctypes

    from paper_1806_01973_amd import _lib
    need = ctypes.c_size_t(0)
    _lib.check(_lib.lib().pinsage_output_mlp_workspace_size(ctypes.byref(mlp.struct()), n,
                                                            ctypes.byref(need)),
               "pinsage_output_mlp_workspace_size")
    return int(need.value)


def ps_mlp(P, wl):
    import torch

    import paper_1806_01973_amd as ps
    return ps.DeviceMLP(P["G1"], P["g"], P["G2"],
                        dtype=torch.bfloat16 if wl.dtype == "bf16" else torch.float32)


def compare_dataflow(args, wl) -> bool:
    if args.pool == "max":
        return False  # max pooling has one order only
    if args.compare_dataflow == "auto":
        return wl.name in ("tiny", "medium")
    return args.compare_dataflow == "on"


def bench_minibatch(args, wl, inp):
    import numpy as np
    import torch

    import paper_1806_01973_amd as ps
    import synth
    B, n_neg = 2048, 500
    k = args.hard_neg or 0
    total = args.steps + args.warmup
    sets = [synth.minibatch_pairs(wl, inp["host"]["offsets"], inp["host"]["col"], B, n_neg,
                                  seed=i) for i in range(total)]
    dev = [[torch.as_tensor(a).cuda() for a in s] for s in sets]
    # The graph's walk table, built once (as a caller would when the graph is
    # loaded): the frontier walks and the hard negatives' walks read it.
    inp["g"].build_walk_table()
    mb = ps.Minibatch(inp["g"], inp["layers"], wl.walks, wl.hops, wl.T, wl.seed, B, n_neg,
                      mlp=inp.get("mlp"), num_hard=k)
    hard = torch.empty((B, k), dtype=torch.int32, device="cuda") if k else None
    stream = torch.cuda.current_stream()
    sizes = []

    def run(i):
        q, p, n = dev[i]
        if k:  # Sec. 3.3: the queries' hard negatives join their negative sets
            ps.hard_negatives(inp["g"], q, k, wl.seed + 1, MB_HN_WALKS, HN_HOPS, HN_LO, HN_HI,
                              out=hard, stream=stream)
        mb.run(inp["x"], q, p, n, 0.1, want_z=False, hard=hard, stream=stream)
        sizes.append(mb.sizes())

    elapsed, prof = timed(run, args.steps, args.warmup)
    kernels = kernel_table(prof, args.steps)
    timed_sizes = np.array(sizes[args.warmup:], dtype=np.float64)
    mean_sizes = timed_sizes.mean(axis=0).tolist()
    value = B * args.steps / elapsed
    # Edge steps of the timed steps' walks (deterministic per minibatch): the
    # timed minibatches again, outside the timed region.
    edge_steps = 0
    for i in range(args.warmup, args.warmup + args.steps):
        run(i)
        edge_steps += int(mb.steps.item())
    edge_steps /= args.steps
    kd = kernels["walk_topt"]
    walk_rates(kd, edge_steps / (kd["launches"] / args.steps), wl.offsets64, table=True)
    inp["g"].drop_walk_table()
    extra = {"walk_steps_per_s": edge_steps / (kd["ms_per_step"] * 1e-3),
             "config_extra": {"pairs": B, "negatives": n_neg, "margin": 0.1,
                              "hard_negatives_per_pair": k, "walk_table": True,
                              "mean_frontier_sizes": mean_sizes,
                              "loss_last": float(mb.loss.item())}}
    metric = ("minibatch forward (Algorithm 2) + max-margin loss, training pairs/sec, 1 MI355X"
              if not k else "hard negative mining (Sec. 3.3) + minibatch forward (Algorithm 2) "
              "+ max-margin loss, training pairs/sec, 1 MI355X")
    return value, "training pairs/s", metric, elapsed, kernels, extra


def cpu_baseline_minibatch(inp, wl, threads, k=0):
    """The oracle's Algorithm 2 route (on-demand neighbourhoods) and Eq. 1 for one
    full minibatch of the same shape (with k hard negatives per pair, mined by
    the oracle first)."""
    import numpy as np
    import oracle
    import synth
    q, p, n = synth.minibatch_pairs(wl, inp["host"]["offsets"], inp["host"]["col"], 2048, 500,
                                    seed=10_000)
    t_hard = time.perf_counter()
    hard = valid = None
    if k:
        hard = oracle.hard_negatives(inp["host"]["offsets"], inp["host"]["col"], wl.num_pins,
                                     wl.seed + 1, MB_HN_WALKS, HN_HOPS, q, HN_LO, HN_HI, k,
                                     nthreads=threads)
        valid = hard >= 0
    t_hard = time.perf_counter() - t_hard
    targets = np.concatenate([q, p, n] + ([hard[valid]] if k else [])).astype("int32")
    t0 = time.perf_counter()
    smp = oracle.minibatch_sample(targets, wl.K, inp["host"]["offsets"], inp["host"]["col"],
                                  wl.num_pins, wl.seed, wl.walks, wl.hops, wl.T, nthreads=threads)
    s0 = smp["sets"][0]
    import torch
    x_rows = inp["x"][torch.as_tensor(s0).long().cuda()].double().cpu().numpy()
    t1 = time.perf_counter()
    z = oracle.minibatch_embed_sampled(targets, s0, x_rows, smp, inp["layers_np"],
                                       nthreads=threads)
    zhard = None
    if k:
        zhard = np.zeros((2048, k, z.shape[1]))
        zhard[valid] = z[4596:]
    oracle.max_margin_loss(z[:2048], z[2048:4096], z[4096:4596], 0.1, zhard, valid)
    t2 = time.perf_counter()
    secs = t_hard + (t1 - t0) + (t2 - t1)
    return {"value": 2048 / secs, "unit": "training pairs/s", "cores": threads, "kind": "oracle",
            "sample": (f"one minibatch of 2048 pairs + 500 negatives"
                       + (f" + {k} hard negatives per pair (mined in {t_hard:.1f}s)" if k else "")
                       + f": on-demand walks {t1 - t0:.1f}s, fp64 Algorithm 2 + Eq. 1 "
                       f"{t2 - t1:.1f}s (feature gather excluded)")}


def bench_hard_negatives(args, wl, inp):
    import numpy as np
    import torch

    import paper_1806_01973_amd as ps
    k = args.hard_neg
    total = args.steps + args.warmup
    rng = np.random.default_rng(wl.seed)
    qs = [torch.as_tensor(rng.integers(0, wl.num_pins, HN_QUERIES).astype(np.int32)).cuda()
          for _ in range(total)]
    out = torch.empty((HN_QUERIES, k), dtype=torch.int32, device="cuda")
    steps_dev = []
    # The graph's walk table, built once (as a caller would when the graph is
    # loaded): every walk step is one dependent read.
    inp["g"].build_walk_table()

    def run(i):
        _, st = ps.hard_negatives(inp["g"], qs[i], k, wl.seed + 1, args.hn_walks, args.hn_hops, HN_LO,
                                  HN_HI, out=out, count_steps=True)
        steps_dev.append(st)

    elapsed, prof = timed(run, args.steps, args.warmup)
    kernels = kernel_table(prof, args.steps)
    edge_steps = sum(int(t.item()) for t in steps_dev[args.warmup:]) / args.steps
    kd = kernels["hard_neg"]
    walk_rates(kd, edge_steps, wl.offsets64, table=True)
    inp["g"].drop_walk_table()
    value = HN_QUERIES * args.steps / elapsed
    extra = {"walk_steps_per_s": edge_steps * args.steps / elapsed,
             "config_extra": {"queries": HN_QUERIES, "walks": args.hn_walks, "hops": args.hn_hops,
                              "rank_window": [HN_LO, HN_HI], "per_query": k, "walk_table": True,
                              "empty_rows_last": int((out[:, 0] < 0).sum().item())}}
    metric = "hard negative items (Sec. 3.3, PPR rank window), queries/sec, 1 MI355X"
    return value, "queries/s", metric, elapsed, kernels, extra


def cpu_baseline_hard_negatives(inp, wl, threads, k, walks=HN_WALKS, hops=HN_HOPS):
    """The oracle's hard negatives for a sample of query pins (16,384 at 4,096 x 4
    landings per query; proportionally fewer at larger budgets: 2,048, one
    step's worth, at the default 32,768 x 4)."""
    import numpy as np
    import oracle
    rng = np.random.default_rng(10_000)
    nq = max(256, 16_384 * 4096 * 4 // (walks * hops))
    q = rng.integers(0, wl.num_pins, nq).astype(np.int32)
    t0 = time.perf_counter()
    oracle.hard_negatives(inp["host"]["offsets"], inp["host"]["col"], wl.num_pins, wl.seed + 1,
                          walks, hops, q, HN_LO, HN_HI, k, nthreads=threads)
    secs = time.perf_counter() - t0
    return {"value": len(q) / secs, "unit": "queries/s", "cores": threads, "kind": "oracle",
            "sample": f"{len(q)} query pins, {secs:.1f}s"}


def layer_probe(args) -> int:
    """One CONVOLVE layer on seeded random inputs, for kernel-level measurement
    (rocprofv3 counters, GEMM tile studies): rows x (d_in, m, d_out) in the
    given dtype and dataflow, T random neighbours per row. Prints per-kernel
    times and rates; not the headline metric."""
    import torch

    import paper_1806_01973_amd as ps
    d_in, m, d_out = (int(v) for v in args.layer.split(","))
    n, T = args.rows, 8
    dt = torch.bfloat16 if args.dtype == "bf16" else torch.float32
    g = torch.Generator(device="cuda").manual_seed(0)
    Q = (torch.randn(m, d_in, device="cuda", generator=g) * 0.05).to(dt)
    W = (torch.randn(d_out, d_in + m, device="cuda", generator=g) * 0.05).to(dt)
    q = torch.zeros(m, device="cuda")
    w = torch.zeros(d_out, device="cuda")
    h = torch.randn(n, d_in, device="cuda", generator=g).to(dt)
    idx = torch.randint(0, n, (n, T), device="cuda", dtype=torch.int32, generator=g)
    cnt = torch.ones((n, T), device="cuda", dtype=torch.int16).view(torch.uint16)
    nb = ps.Neighborhoods(idx, cnt, None)
    L = ps.DeviceLayer(Q, q, W, w, dtype=dt, dataflow=args.dataflow)
    ws = torch.empty(ps.convolve_workspace_size(L, n, n), dtype=torch.uint8, device="cuda")
    out = torch.empty((n, d_out), dtype=dt, device="cuda")
    steps = args.steps if args.steps is not None else 3
    _, prof = timed(lambda i: ps.convolve_layer(L, h, n, nb, out=out, workspace=ws),
                    steps, args.warmup if args.warmup is not None else 1)
    peak = MFMA_PEAK_TFLOPS[args.dtype]
    split = args.dataflow == "dense_then_pool"
    flops = {"gemm_q": 2.0 * n * d_in * m, "gemm_r": 2.0 * n * m * d_out if split else 0.0,
             "gemm_w": 2.0 * n * (d_in + (0 if split else m)) * d_out}
    res = {"layer": [d_in, m, d_out], "rows": n, "dtype": args.dtype, "dataflow": args.dataflow}
    for name, (launches, ms) in prof.items():
        if launches and name in flops:
            per_call = ms / steps
            res[name] = {"ms": per_call, "TFLOP/s": flops[name] / (per_call * 1e-3) / 1e12,
                         "frac_mfma": flops[name] / (per_call * 1e-3) / 1e12 / peak}
        elif launches:
            res[name] = {"ms": ms / steps}
    if args.blas_ref:
        res["blas_reference"] = blas_reference(n, [(d_in, m), (m, d_out)], dt, peak)
    print(json.dumps(res), flush=True)
    return 0


def blas_reference(n, shapes, dt, peak):
    """Library GEMM rates (torch.matmul, i.e. hipBLASLt) for the plain products
    [n, K] x [K, N] of the given (K, N) shapes, without bias or epilogue: a
    reference point for the layer GEMMs, not part of the path."""
    import torch
    out = {}
    for K, N in shapes:
        a = torch.randn(n, K, device="cuda").to(dt)
        b = torch.randn(N, K, device="cuda").to(dt)
        bt = b.t()
        for _ in range(2):
            c = a @ bt
        torch.cuda.synchronize()
        s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        s.record()
        for _ in range(5):
            c = a @ bt
        e.record()
        torch.cuda.synchronize()
        ms = s.elapsed_time(e) / 5
        tf = 2.0 * n * K * N / (ms * 1e-3) / 1e12
        out[f"{n}x{K}x{N}"] = {"ms": ms, "TFLOP/s": tf, "frac_mfma": tf / peak}
        del a, b, bt, c
        torch.cuda.empty_cache()
    return out


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None)
    ap.add_argument("--warmup", type=int, default=None)
    ap.add_argument("--workload", default="shard",
                    choices=["tiny", "medium", "minibatch", "large", "shard", "hardneg",
                             "bipartite"])
    ap.add_argument("--dataflow", default="dense_then_pool",
                    choices=["pool_then_dense", "dense_then_pool"],
                    help="layer evaluation order (same values; see pinsage_dataflow_t)")
    ap.add_argument("--compare-dataflow", default="auto", choices=["auto", "on", "off"],
                    help="also time the other evaluation order (auto: small workloads)")
    ap.add_argument("--pool", default="importance", choices=["importance", "mean", "max"],
                    help="aggregator of every layer (max implies the pool-then-dense order)")
    ap.add_argument("--mlp", type=int, default=0, metavar="D_HIDDEN",
                    help="append the output dense layers z = G2 ReLU(G1 h + g) to the step")
    ap.add_argument("--hard-neg", type=int, default=None, metavar="K",
                    help="hard negatives per query: draws for --workload hardneg (default 4); "
                         "with --workload minibatch, mined each step and added to every "
                         "pair's negatives (default 0)")
    ap.add_argument("--hn-walks", type=int, default=HN_WALKS,
                    help="--workload hardneg: walks per query (walks x hops above 16,384 "
                         "count visits in a global table)")
    ap.add_argument("--hn-hops", type=int, default=HN_HOPS,
                    help="--workload hardneg: pin landings per walk")
    ap.add_argument("--overlap", type=int, default=4, metavar="EIGHTHS",
                    help="all-node job: first layer's transform beside the walks on EIGHTHS/8 "
                         "of the CUs (0: walks, then transform, in order)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--layer", default=None,
                    help="d_in,m,d_out: time one layer on random inputs instead of a workload")
    ap.add_argument("--rows", type=int, default=4_000_000, help="rows for --layer")
    ap.add_argument("--dtype", default="bf16", choices=["bf16", "f32"], help="dtype for --layer")
    ap.add_argument("--blas-ref", action="store_true",
                    help="with --layer: also time torch.matmul on the layer's GEMM shapes")
    ap.add_argument("--copy-calibration", action="store_true")
    ap.add_argument("--random-read-calibration", action="store_true",
                    help="dependent random reads/s from a 16 GiB table (the walks' ceiling)")
    ap.add_argument("--gather-calibration", action="store_true",
                    help="random 512-byte and 1 KB row gathers/s in the pool's pattern (the "
                         "pool's ceiling)")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the path runs on a single MI355X and has no "
              "multi-GPU mode; run it with --gpus 1.", file=sys.stderr)
        return 2

    import torch

    if args.copy_calibration:
        copy_calibration()
        return 0
    if args.random_read_calibration:
        random_read_calibration()
        return 0
    if args.gather_calibration:
        random_gather_calibration()
        return 0
    if args.layer:
        return layer_probe(args)

    import synth

    hardneg = args.workload == "hardneg"
    bipartite = args.workload == "bipartite"
    if hardneg and args.hard_neg is None:
        args.hard_neg = 4
    wl = synth.WORKLOADS["medium" if hardneg or bipartite else args.workload]
    args.steps = args.steps if args.steps is not None else DEFAULT_STEPS[args.workload]
    args.warmup = args.warmup if args.warmup is not None else DEFAULT_WARMUP[args.workload]
    if args.pool == "max" and args.dataflow == "dense_then_pool":
        args.dataflow = "pool_then_dense"  # max pooling is not linear
    inp = load_inputs(wl, args.dataflow, args.pool)
    if args.mlp:
        import synth as _s
        P = _s.make_mlp(wl.d_out, args.mlp, wl.d_out, seed=wl.seed, dtype=wl.dtype)
        inp["mlp"] = ps_mlp(P, wl)
    if hardneg:
        value, unit, metric, elapsed, kernels, extra = bench_hard_negatives(args, wl, inp)
    elif bipartite:
        value, unit, metric, elapsed, kernels, extra = bench_bipartite(args, wl, inp)
    elif wl.name == "minibatch":
        value, unit, metric, elapsed, kernels, extra = bench_minibatch(args, wl, inp)
    else:
        value, unit, metric, elapsed, kernels, extra = bench_embed_all(args, wl, inp)

    result = {
        "metric": metric,
        "value": value,
        "unit": unit,
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": 1e3 * elapsed / args.steps,
        "ms_per_step_median": (sorted(STEP_MS)[len(STEP_MS) // 2] if STEP_MS else None),
        "ms_per_step_each": [round(t, 3) for t in STEP_MS],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u32" if hardneg else wl.dtype,
        "data": "synthetic",
        "config": {"workload": (f"hard negatives: {wl.num_pins} pins + {wl.num_boards} boards, "
                                f"{inp['num_edges']} edges, {HN_QUERIES} query pins, {args.hn_walks} "
                                f"walks x {args.hn_hops} landings each, ranks {HN_LO + 1}-{HN_HI}, "
                                f"{args.hard_neg} per query") if hardneg else
                   (f"{wl.name}: {wl.num_pins} pins + {wl.num_boards} boards, "
                               f"{inp['num_edges']} edges, {wl.walks} walks x {wl.hops} hops, "
                               f"T={wl.T}, K={wl.K}, dims {wl.d_in}->{wl.m}->{wl.d_out} "
                               f"{wl.dtype}, layer dataflow {args.dataflow}"
                               + (f", pool {args.pool}" if args.pool != "importance" else "")
                               + (f", output layers {wl.d_out}->{args.mlp}->{wl.d_out}"
                                  if args.mlp else "")),
                   "dataflow": args.dataflow, "pool": args.pool, "output_layers": args.mlp or None,
                   "edges": inp["num_edges"], "gpu": torch.cuda.get_device_name(0),
                   **extra["config_extra"]},
        "walk_steps_per_s": extra["walk_steps_per_s"],
        "walk_steps_per_s_all_cus": extra.get("walk_steps_per_s_all_cus"),
        "layers_embeddings_per_s": extra.get("layers_embeddings_per_s"),
        "alt_dataflow": extra.get("alt_dataflow"),
        "roofline": roofline_of(kernels, wl),
        "kernels": kernels,
        "cpu_baseline": None,
    }
    if bipartite:
        result["config"]["workload"] = (
            f"MapReduce inference variant on {wl.name}: {wl.num_pins} pins + {wl.num_boards} "
            f"boards, {inp['num_edges']} edges, graph neighbourhoods T={wl.T} (longer rows "
            f"sampled), featureless boards, K={wl.K}, dims {wl.d_in}->{wl.m}->{wl.d_out} "
            f"{wl.dtype}, layer dataflow {args.dataflow}")
    if not args.no_cpu_baseline:
        import oracle
        threads = oracle.default_threads()
        log(f"timing the oracle on a sample ({threads} threads)")
        if hardneg:
            result["cpu_baseline"] = cpu_baseline_hard_negatives(inp, wl, threads, args.hard_neg,
                                                                 args.hn_walks, args.hn_hops)
        elif bipartite:
            result["cpu_baseline"] = cpu_baseline_bipartite(inp, wl, threads)
        elif wl.name == "minibatch":
            result["cpu_baseline"] = cpu_baseline_minibatch(inp, wl, threads,
                                                            args.hard_neg or 0)
        else:
            result["cpu_baseline"] = cpu_baseline_embed(inp, wl, threads)
        result["cpu_baseline"]["host"] = host_cpu()
    print(json.dumps(result), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
