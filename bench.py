"""Benchmark: all-node PinSage embedding on one MI355X.

One step = the whole hot path over the 1.2M-node pin-board workload (1M pins,
200k boards, fp32, dims 256 -> 512 -> 256, 100 walks x 3 hops, T = 50):
importance neighbourhoods of every node, then K = 2 CONVOLVE layers over every
node, layer by layer. Inputs are resident in HBM before timing starts.

Prints one JSON line: node embeddings/s for the whole step (the headline),
walk steps/s, per-kernel times from hipEvents recorded around every launch in
the timed region, the roofline of the dominant kernel and the CPU oracle timed
on a bounded sample of the same workload.

  python bench.py [--steps K] [--warmup W] [--workload medium] [--no-cpu-baseline]
  python bench.py --copy-calibration   # plain copy of a known size, for counter scaling
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


def log(msg: str) -> None:
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def kernel_source_hash(name: str) -> str:
    path = os.path.join(ROOT, "paper_1806_01973_amd", "csrc", name)
    with open(path, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


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


def cpu_baseline(data, wl, threads: int) -> dict:
    """The oracle as it stands, on a bounded sample of the same workload:
    neighbourhoods of a node sample, and each layer on a row sample (pins
    projected in the same pin:node proportion). Extrapolated per node."""
    import numpy as np
    import oracle

    n_walk = 400_000
    n_rows = 120_000
    N, P = wl.num_nodes, wl.num_pins
    rng = np.random.default_rng(123)
    src = np.sort(rng.choice(N, n_walk, replace=False)).astype(np.int32)
    t0 = time.perf_counter()
    idx, cnt, wts, steps = oracle.build_neighborhoods(data["offsets"], data["col"], P, wl.seed,
                                                      wl.walks, wl.hops, wl.T, sources=src,
                                                      nthreads=threads)
    t_walk = time.perf_counter() - t0
    # Layer sample: rows [0, n_rows) of the node features, n_transform pins
    # among them, neighbour ids folded into that range.
    n_tr = int(round(n_rows * P / N))
    idx_s = np.where(idx[:n_rows] >= 0, idx[:n_rows] % n_tr, -1).astype(np.int32)
    wts_s = wts[:n_rows]
    h = data["x"][:n_rows]
    t_layers = 0.0
    for L in data["layers"]:
        t0 = time.perf_counter()
        h = oracle.convolve_layer(h, n_tr, L["Q"], L["q"], L["W"], L["w"], idx_s, wts_s,
                                  nthreads=threads)
        t_layers += time.perf_counter() - t0
    per_node = t_walk / n_walk + t_layers / n_rows
    return {"value": 1.0 / per_node, "unit": "node embeddings/s", "cores": threads,
            "kind": "oracle",
            "sample": (f"neighbourhoods of {n_walk} random nodes ({t_walk:.1f}s, "
                       f"{steps / t_walk:.3g} walk steps/s) + both layers on {n_rows} rows "
                       f"with {n_tr} projected pins ({t_layers:.1f}s), fp64, extrapolated "
                       f"per node"),
            "walk_steps_per_s": steps / t_walk}


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="medium")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration", action="store_true")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the path runs on a single MI355X and has no "
              "multi-GPU mode; run it with --gpus 1.", file=sys.stderr)
        return 2

    import numpy as np
    import torch

    if args.copy_calibration:
        copy_calibration()
        return 0

    import paper_1806_01973_amd as ps
    import synth

    wl = synth.WORKLOADS[args.workload]
    t0 = time.perf_counter()
    data = synth.make_workload(wl)
    log(f"generated {wl.name}: {wl.num_nodes} nodes, {data['num_edges']} edges "
        f"in {time.perf_counter() - t0:.1f}s")
    tdt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    g = ps.DeviceGraph(data["offsets"], data["col"], wl.num_pins, wl.num_boards,
                       offsets64=wl.offsets64)
    layers = [ps.DeviceLayer(L["Q"], L["q"], L["W"], L["w"], dtype=tdt) for L in data["layers"]]
    x = torch.as_tensor(data["x"]).to(device="cuda", dtype=tdt)
    job = ps.EmbedAll(g, layers, wl.walks, wl.hops, wl.T, wl.seed)
    stream = torch.cuda.current_stream()

    for _ in range(args.warmup):
        job.run(x, stream)
    torch.cuda.synchronize()
    log(f"warmup done ({args.warmup} steps)")

    ps.profile_enable(True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        job.run(x, stream)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    prof = ps.profile_read()
    ps.profile_enable(False)
    log(f"timed {args.steps} steps in {elapsed:.3f}s")

    N = wl.num_nodes
    steps_per_run = int(job.steps.item())
    ms_per_step = 1e3 * elapsed / args.steps
    value = N * args.steps / elapsed

    # Algorithmic work per launch.
    esz = 2 if wl.dtype == "bf16" else 4
    live = (job.nbr.idx >= 0).sum().item()
    idx_bytes = N * wl.T * 4 + (N * wl.T * 4 if job.nbr.weights is not None else N * wl.T * 2)
    pool_bytes = [live * L.m * esz + idx_bytes + N * L.m * esz for L in layers]
    gq_flops = [2.0 * wl.num_pins * L.d_in * L.m for L in layers]
    gw_flops = [2.0 * N * (L.d_in + L.m) * L.d_out for L in layers]
    off_b = 8 if wl.offsets64 else 4
    walk_bytes = steps_per_run * (2 * off_b + 4)

    kernels = {}
    for name, (n_launch, ms) in prof.items():
        if n_launch == 0:
            continue
        kernels[name] = {"launches": n_launch, "avg_ms": ms / n_launch,
                         "ms_per_step": ms / args.steps}
    # Pool: algorithmic bytes per launch (both layers alike when m is equal).
    pool_avg_bytes = sum(pool_bytes) / len(pool_bytes)
    if "pool" in kernels:
        k = kernels["pool"]
        k["algo_bytes_per_launch"] = pool_avg_bytes
        k["achieved_GBs"] = pool_avg_bytes / (k["avg_ms"] * 1e-3) / 1e9
        k["frac_hbm"] = k["achieved_GBs"] / HBM_PEAK_GBS
    peak_tf = MFMA_PEAK_TFLOPS[wl.dtype]
    for name, fl in (("gemm_q", gq_flops), ("gemm_w", gw_flops)):
        if name in kernels:
            k = kernels[name]
            k["algo_flops_per_launch"] = sum(fl) / len(fl)
            k["achieved_TFLOPs"] = k["algo_flops_per_launch"] / (k["avg_ms"] * 1e-3) / 1e12
            k["frac_mfma"] = k["achieved_TFLOPs"] / peak_tf
    walk_steps_per_s = None
    if "walk_topt" in kernels:
        k = kernels["walk_topt"]
        k["edge_steps_per_launch"] = steps_per_run
        k["algo_bytes_per_launch"] = walk_bytes
        k["achieved_GBs"] = walk_bytes / (k["avg_ms"] * 1e-3) / 1e9
        walk_steps_per_s = steps_per_run / (k["avg_ms"] * 1e-3)

    dominant = max(kernels, key=lambda n: kernels[n]["ms_per_step"])
    kd = kernels[dominant]
    if dominant in ("gemm_q", "gemm_w"):
        roof = {"kernel": dominant, "bound": "mfma", "achieved": kd["achieved_TFLOPs"],
                "peak": peak_tf, "unit": "TFLOP/s", "frac": kd["frac_mfma"], "traffic": None}
    else:
        src_file = {"pool": "pool.hip", "walk_topt": "walk.hip"}[dominant]
        tr = load_traffic(src_file, wl.name)
        roof = {"kernel": dominant, "bound": "hbm", "achieved": kd["achieved_GBs"],
                "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": kd["achieved_GBs"] / HBM_PEAK_GBS,
                "traffic": None if tr is None else tr["bytes_per_launch"]}

    result = {
        "metric": METRIC,
        "value": value,
        "unit": "node embeddings/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": wl.dtype,
        "data": "synthetic",
        "config": {"workload": f"{wl.name}: {wl.num_pins} pins + {wl.num_boards} boards, "
                               f"{data['num_edges']} edges, {wl.walks} walks x {wl.hops} hops, "
                               f"T={wl.T}, K={wl.K}, dims {wl.d_in}->{wl.m}->{wl.d_out} "
                               f"{wl.dtype}",
                   "nodes": N, "edges": int(data["num_edges"]), "walk_steps_per_step": steps_per_run,
                   "gpu": torch.cuda.get_device_name(0)},
        "walk_steps_per_s": walk_steps_per_s,
        "roofline": roof,
        "kernels": kernels,
        "cpu_baseline": None,
    }
    if not args.no_cpu_baseline:
        import oracle
        threads = oracle.default_threads()
        log(f"timing the oracle on a sample ({threads} threads)")
        result["cpu_baseline"] = cpu_baseline(data, wl, threads)
    print(json.dumps(result), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
