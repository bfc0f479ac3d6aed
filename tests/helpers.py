"""Shared test helpers: tolerance checks and input staging.

Tolerances (per element, o = oracle value in fp64, g = GPU value):
    |g - o| <= rtol * (|o| + 1/sqrt(d))
with rtol = 1e-4 for fp32 storage and 2e-2 for bf16 storage, plus a per-row
cosine >= 0.999 for bf16. 1/sqrt(d) is the RMS entry of a unit vector in d
dimensions; it keeps the relative test meaningful at entries that ReLU sets to
(or near) zero. The stats count the elements that pass only because of that
absolute part ("floor_only").
"""

from __future__ import annotations

import numpy as np

RTOL = {"f32": 1e-4, "bf16": 2e-2}


def check_embeddings(got: np.ndarray, ref: np.ndarray, dtype: str, what: str = "") -> dict:
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    d = ref.shape[1]
    rtol = RTOL[dtype]
    bound = rtol * (np.abs(ref) + 1.0 / np.sqrt(d))
    err = np.abs(got - ref)
    bad = err > bound
    worst = float((err / bound).max()) if err.size else 0.0
    assert not bad.any(), (f"{what}: {int(bad.sum())} of {bad.size} elements outside tolerance; "
                           f"worst err/bound = {worst:.3g} at {np.unravel_index(np.argmax(err / bound), err.shape)}")
    # Elements inside the bound only thanks to its absolute part rtol/sqrt(d)
    # (entries at or near a ReLU zero): counted and reported so that a drift
    # of the small entries stays visible.
    floor_only = int(((err > rtol * np.abs(ref)) & ~bad).sum())
    stats = {"max_err_over_bound": worst, "elements": int(err.size),
             "floor_only": floor_only}
    if dtype == "bf16":
        ng = np.linalg.norm(got, axis=1)
        nr = np.linalg.norm(ref, axis=1)
        live = (nr > 0) & (ng > 0)
        cos = (got[live] * ref[live]).sum(1) / (ng[live] * nr[live])
        assert np.all(cos >= 0.999), f"{what}: min cosine {cos.min():.6f}"
        stats["min_cos"] = float(cos.min()) if cos.size else 1.0
    return stats


def to_f64(t) -> np.ndarray:
    import torch
    return t.detach().to(device="cpu", dtype=torch.float64).numpy()


def torch_dtype(dtype: str):
    import torch
    return torch.bfloat16 if dtype == "bf16" else torch.float32
