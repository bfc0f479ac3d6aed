"""Host-side logic of bench.py (no GPU): the per-kernel table, the algorithmic
work per launch behind the roofline, the choice of the dominant kernel, the
counter-summary lookup keyed by the kernel's source hash, and the one-GPU
refusal of --gpus N > 1."""

import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
import synth  # noqa: E402


class _Layer:
    def __init__(self, d_in, m, d_out, dataflow, dtype=None):
        self.d_in, self.m, self.d_out, self.dataflow = d_in, m, d_out, dataflow
        self.dtype = dtype


def _medium_kernels():
    # Two timed steps of the 1.2M-node job: per step one walk, two launches of
    # each layer kernel (hipEvent totals in ms).
    prof = {"walk_topt": (2, 20.0), "pool": (4, 26.0), "gemm_q": (4, 10.0),
            "gemm_r": (4, 9.0), "gemm_w": (4, 6.0), "loss": (0, 0.0)}
    return bench.kernel_table(prof, 2)


def test_kernel_table():
    k = _medium_kernels()
    assert "loss" not in k
    assert k["pool"] == {"launches": 4, "avg_ms": 6.5, "ms_per_step": 13.0}
    assert k["walk_topt"]["ms_per_step"] == 10.0


def test_algorithmic_work_per_launch():
    wl = synth.WORKLOADS["medium"]
    N, P = wl.num_nodes, wl.num_pins
    layers = [_Layer(256, 512, 256, "dense_then_pool")] * 2
    k = _medium_kernels()
    live, steps = 53_815_669, 639_125_000
    bench.add_rooflines(k, wl, layers, N, P, live, True, steps, 2)
    # Pool: gathered d_out-wide fp32 rows + idx and weights + the written rows, per layer.
    per_layer = live * 256 * 4 + N * wl.T * 8 + N * 256 * 4
    assert k["pool"]["algo_bytes_per_launch"] == pytest.approx(per_layer)
    assert k["pool"]["achieved_GBs"] == pytest.approx(per_layer / 6.5e-3 / 1e9)
    # GEMMs: 2 P d_in m (Q), 2 P m d_out (R), 2 N d_in d_out (W, dense then pool).
    assert k["gemm_q"]["algo_flops_per_launch"] == pytest.approx(2.0 * P * 256 * 512)
    assert k["gemm_r"]["algo_flops_per_launch"] == pytest.approx(2.0 * P * 512 * 256)
    assert k["gemm_w"]["algo_flops_per_launch"] == pytest.approx(2.0 * N * 256 * 256)
    assert k["gemm_w"]["frac_mfma"] == pytest.approx(
        2.0 * N * 256 * 256 / 1.5e-3 / 1e12 / 157.3)
    # Walk: 12 B per edge step with int32 row offsets.
    assert k["walk_topt"]["algo_bytes_per_launch"] == pytest.approx(steps * 12)
    # Pool then dense: the pool gathers m-wide rows and W has K = d_in + m.
    k2 = _medium_kernels()
    del k2["gemm_r"]
    bench.add_rooflines(k2, wl, [_Layer(256, 512, 256, "pool_then_dense")] * 2, N, P, live,
                        True, steps, 2)
    assert k2["pool"]["algo_bytes_per_launch"] == pytest.approx(
        live * 512 * 4 + N * wl.T * 8 + N * 512 * 4)
    assert k2["gemm_w"]["algo_flops_per_launch"] == pytest.approx(2.0 * N * 768 * 256)


def test_dominant_kernel_roofline_and_traffic(monkeypatch, tmp_path):
    # Counter bytes of the current pool source are reported as `traffic`.
    (tmp_path / "traffic.json").write_text(json.dumps(
        {"pool.hip:medium": {"source_sha": bench.kernel_source_hash("pool.hip"),
                             "bytes_per_launch": 4.5e10, "profile": "profiles/x.md"}}))
    monkeypatch.setattr(bench, "PROFILE_DIR", str(tmp_path))
    wl = synth.WORKLOADS["medium"]
    k = _medium_kernels()
    bench.add_rooflines(k, wl, [_Layer(256, 512, 256, "dense_then_pool")] * 2,
                        wl.num_nodes, wl.num_pins, 53_815_669, True, 639_125_000, 2)
    r = bench.roofline_of(k, wl)
    assert r["kernel"] == "pool" and r["bound"] == "hbm" and r["unit"] == "GB/s"
    assert r["peak"] == 8000.0 and r["frac"] == pytest.approx(r["achieved"] / 8000.0)
    assert r["traffic"] == 4.5e10
    assert r["traffic_GBs"] == pytest.approx(4.5e10 / (k["pool"]["avg_ms"] * 1e-3) / 1e9)
    assert r.get("cache_resident", False) == (r["frac"] > 1.0)
    # A GEMM-dominated step reports the MFMA roofline for its dtype and no traffic.
    k["gemm_q"]["ms_per_step"] = 100.0
    r = bench.roofline_of(k, wl)
    assert r["kernel"] == "gemm_q" and r["bound"] == "mfma" and r["peak"] == 157.3
    assert r["traffic"] is None


def test_walk_bound_roofline():
    # A walk-dominated line (the hard negative bench) labels its algorithmic
    # bytes as the edge steps' reads and carries the random-read floor.
    k = {"hard_neg": {"ms_per_step": 12.9, "avg_ms": 12.9}}
    bench.walk_rates(k["hard_neg"], 536_870_912, False, table=True)
    r = bench.roofline_of(k, synth.WORKLOADS["medium"])
    assert r["kernel"] == "hard_neg" and r["bound"] == "hbm"
    assert "walk-table entry" in r["bytes"]
    assert r["achieved"] == pytest.approx(536_870_912 * 16 / (12.9e-3) / 1e9)
    assert r["random_read_floor_ms"] == pytest.approx(536_870_912 / bench.RANDOM_READS_PER_S * 1e3)
    assert r["frac_of_random_read_floor"] == pytest.approx(r["random_read_floor_ms"] / 12.9)


def test_counter_summaries_match_current_sources():
    # Every committed counter summary was taken on the kernel source now in the
    # tree (else the bench reports no traffic for it, and the summary is stale).
    with open(os.path.join(ROOT, "profiles", "traffic.json")) as f:
        table = json.load(f)
    for key, ent in table.items():
        src = key.split(":")[0]
        assert ent["source_sha"] == bench.kernel_source_hash(src), key
        assert os.path.exists(os.path.join(ROOT, ent["profile"])), key


def test_stale_source_gives_no_traffic(monkeypatch, tmp_path):
    (tmp_path / "traffic.json").write_text(json.dumps(
        {"pool.hip:medium": {"source_sha": "0000000000000000", "bytes_per_launch": 1.0,
                             "profile": "x"}}))
    monkeypatch.setattr(bench, "PROFILE_DIR", str(tmp_path))
    assert bench.load_traffic("pool.hip", "medium") is None
    assert bench.load_traffic("walk.hip", "medium") is None


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in (r.stdout + r.stderr)


def test_chained_transform_accounting():
    # bf16 dense-then-pool layers of 256 -> 512 -> 256 run the Q transform and
    # the neighbour half of W as one kernel: its flops are both products'.
    import torch
    wl = synth.WORKLOADS["shard"]
    N, P = wl.num_nodes, wl.num_pins
    layers = [_Layer(256, 512, 256, "dense_then_pool", torch.bfloat16)] * 2
    k = {"gemm_qr": {"launches": 2, "avg_ms": 40.0, "ms_per_step": 80.0},
         "gemm_w": {"launches": 48, "avg_ms": 1.9, "ms_per_step": 91.2}}
    bench.add_rooflines(k, wl, layers, N, P, 0, False, 0, 1)
    assert k["gemm_qr"]["algo_flops_per_launch"] == pytest.approx(
        2.0 * P * (256 * 512 + 512 * 256))
    assert k["gemm_qr"]["frac_mfma"] == pytest.approx(
        k["gemm_qr"]["algo_flops_per_launch"] / 40e-3 / 1e12 / 2500.0)
    assert "gemm_q" not in k and "gemm_r" not in k
    assert not bench.chained_layer(_Layer(256, 512, 256, "pool_then_dense", torch.bfloat16))
    assert not bench.chained_layer(_Layer(1024, 2048, 512, "dense_then_pool", torch.bfloat16))


def test_walk_rates_csr_and_table():
    steps = 1e9
    csr = {"avg_ms": 100.0}
    bench.walk_rates(csr, steps, offsets64=True)
    assert csr["algo_bytes_per_launch"] == steps * 20  # offset pair (2 x 8 B) + id
    assert csr["transaction_floor_ms"] == pytest.approx(steps * 128 / 8e12 * 1e3)
    tab = {"avg_ms": 100.0}
    bench.walk_rates(tab, steps, offsets64=True, table=True)
    assert tab["walk_table"] and not csr["walk_table"]
    assert tab["algo_bytes_per_launch"] == steps * 16  # one table entry
    assert tab["transaction_floor_ms"] == pytest.approx(steps * 64 / 8e12 * 1e3)
    rr = steps / bench.RANDOM_READS_PER_S * 1e3
    assert tab["random_read_floor_ms"] == pytest.approx(rr)
    assert tab["frac_of_random_read_floor"] == pytest.approx(rr / 100.0)
