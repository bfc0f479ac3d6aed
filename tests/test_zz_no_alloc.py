"""GPU: pinsage_convolve_layer_noalloc (the convolve layer whose workspace is
the library's static per-GPU scratch, for callers that cannot allocate)
against pinsage_convolve_layer with a caller workspace, both called through
the C ABI on the same seeded inputs. The two share every kernel and the
chunking of rows, so the outputs must agree bit for bit; each case runs two
calls in a row, the second on a smaller input (the scratch then holds the
first call's contents), in fp32 and bf16 storage and in both layer dataflows.
A layer whose workspace exceeds the scratch is refused before any launch.
"""

import ctypes

import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

DIMS = (256, 512, 256)  # d_in, m, d_out of the 256 -> 512 -> 256 workloads


def _inputs(rng, n_in, n_transform, n_out, T, dt):
    """Seeded rows, parameters and a neighbourhood table with padded tails."""
    import paper_1806_01973_amd as ps
    d_in, m, d_out = DIMS
    h = torch.as_tensor(rng.standard_normal((n_in, d_in)), dtype=torch.float32)
    lim_q = np.sqrt(6.0 / (d_in + m))
    lim_w = np.sqrt(6.0 / (d_in + m + d_out))
    Q = torch.as_tensor(rng.uniform(-lim_q, lim_q, (m, d_in)), dtype=torch.float32)
    W = torch.as_tensor(rng.uniform(-lim_w, lim_w, (d_out, d_in + m)), dtype=torch.float32)
    q = torch.as_tensor(rng.uniform(-0.1, 0.1, m), dtype=torch.float32)
    w = torch.as_tensor(rng.uniform(-0.1, 0.1, d_out), dtype=torch.float32)
    idx = rng.integers(0, n_transform, (n_out, T)).astype(np.int32)
    live = rng.integers(0, T + 1, n_out)  # live slots per row, rest padding
    cnt = rng.integers(1, 20, (n_out, T)).astype(np.uint16)
    pad = np.arange(T)[None, :] >= live[:, None]
    idx[pad] = -1
    cnt[pad] = 0
    nb = ps.Neighborhoods(torch.as_tensor(idx).cuda(),
                          torch.as_tensor(cnt.view(np.int16)).cuda().view(torch.uint16), None)
    return h.to(dt).cuda(), (Q.to(dt).cuda(), q.cuda(), W.to(dt).cuda(), w.cuda()), nb


def _call(fn_name, layer, h, n_transform, nb, out, ws=None):
    from paper_1806_01973_amd import _lib as L
    lib = L.lib()
    ns = nb.struct()
    ls = layer.struct()
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    if fn_name == "pinsage_convolve_layer":
        st = lib.pinsage_convolve_layer(ctypes.byref(ls), h.data_ptr(), h.shape[0], n_transform,
                                        None, ctypes.byref(ns), None, out.data_ptr(), nb.rows,
                                        ws.data_ptr(), ws.numel(), stream)
    else:
        st = lib.pinsage_convolve_layer_noalloc(ctypes.byref(ls), h.data_ptr(), h.shape[0],
                                                n_transform, None, ctypes.byref(ns), None,
                                                out.data_ptr(), nb.rows, stream)
    return st


@pytest.mark.parametrize("dtype,dataflow,sizes", [
    ("f32", "pool_then_dense", [(14_000, 11_000, 13_000), (3_001, 2_500, 2_999)]),
    ("f32", "dense_then_pool", [(16_000, 12_000, 14_000), (4_097, 4_000, 1_000)]),
    ("bf16", "pool_then_dense", [(30_000, 25_000, 29_000), (700, 500, 640)]),
    ("bf16", "dense_then_pool", [(33_000, 30_000, 32_000), (5_000, 4_100, 4_999)]),
])
def test_noalloc_matches_workspace_entry_point(dtype, dataflow, sizes):
    import paper_1806_01973_amd as ps
    from paper_1806_01973_amd import _lib as L
    dt = torch.bfloat16 if dtype == "bf16" else torch.float32
    rng = np.random.default_rng(77)
    for call, (n_in, n_transform, n_out) in enumerate(sizes):
        print(f"[case] noalloc {dtype} {dataflow} call {call}: n_in={n_in} "
              f"n_transform={n_transform} n_out={n_out}", flush=True)
        h, (Q, q, W, w), nb = _inputs(rng, n_in, n_transform, n_out, 50, dt)
        layer = ps.DeviceLayer(Q, q, W, w, dtype=dt, dataflow=dataflow)
        need = ps.convolve_workspace_size(layer, n_transform, n_out)
        assert need <= (64 << 20), need
        ws = torch.empty(need, dtype=torch.uint8, device="cuda")
        ref = torch.empty((n_out, DIMS[2]), dtype=dt, device="cuda")
        got = torch.full((n_out, DIMS[2]), 7.0, dtype=dt, device="cuda")
        assert _call("pinsage_convolve_layer", layer, h, n_transform, nb, ref, ws) == 0
        st = _call("pinsage_convolve_layer_noalloc", layer, h, n_transform, nb, got)
        assert st == 0, L.lib().pinsage_last_error()
        torch.cuda.synchronize()
        assert torch.isfinite(ref.float()).all()
        assert torch.equal(got, ref), f"call {call}: outputs differ"
        norms = torch.linalg.vector_norm(got.float(), dim=1)
        tol = 1e-2 if dtype == "bf16" else 1e-5
        assert torch.all(((norms - 1).abs() < tol) | (norms == 0))


def test_noalloc_refuses_layers_beyond_the_scratch():
    import paper_1806_01973_amd as ps
    from paper_1806_01973_amd import _lib as L
    rng = np.random.default_rng(5)
    n_in, n_transform, n_out = 70_000, 60_000, 70_000
    h, (Q, q, W, w), nb = _inputs(rng, n_in, n_transform, n_out, 8, torch.float32)
    layer = ps.DeviceLayer(Q, q, W, w, dtype=torch.float32, dataflow="pool_then_dense")
    assert ps.convolve_workspace_size(layer, n_transform, n_out) > (64 << 20)
    out = torch.zeros((n_out, DIMS[2]), device="cuda")
    print("[case] noalloc beyond the scratch", flush=True)
    st = _call("pinsage_convolve_layer_noalloc", layer, h, n_transform, nb, out)
    assert st == L.PINSAGE_EUNSUPPORTED
    assert b"scratch" in L.lib().pinsage_last_error()
    torch.cuda.synchronize()
    assert torch.count_nonzero(out) == 0  # nothing launched
