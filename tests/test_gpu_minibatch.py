"""GPU parity: minibatch forward (Algorithm 2) and the max-margin loss (Eq. 1).

* The loss kernel against the oracle on generator-made unit vectors.
* The whole minibatch forward -- frontier sets, on-device re-indexing, both
  layers on the compact sets, loss -- against the oracle's Algorithm 2 run on
  the oracle's own neighbourhood table: frontier sizes exactly, target
  embeddings to the storage dtype's tolerance, and the loss to the bound that
  the observed embedding errors imply (the hinge is 1-Lipschitz, so
  |loss_gpu - loss_oracle| <= mean over pairs of the dot-product errors, each
  bounded by |da|.|b| + |a|.|db| + |da|.|db|).
"""

import numpy as np
import pytest
import torch

import synth
from helpers import check_embeddings, to_f64, torch_dtype

pytestmark = pytest.mark.gpu


def _unit_rows(rng, n, d):
    z = rng.standard_normal((n, d))
    return (z / np.linalg.norm(z, axis=1, keepdims=True)).astype(np.float32)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("B,n_neg,d", [(333, 77, 200), (2048, 500, 256), (37, 301, 512),
                                       (19, 45, 1024), (5, 3, 13)])
def test_loss_kernel(orc, dtype, B, n_neg, d):
    import paper_1806_01973_amd as ps
    rng = np.random.default_rng(3)
    zq, zp, zn = _unit_rows(rng, B, d), _unit_rows(rng, B, d), _unit_rows(rng, n_neg, d)
    # Make some pairs hard so the hinge is active for a mix of negatives.
    hard = min(100, B // 3)
    zp[:hard] = zq[:hard] * 0.3 + zp[:hard] * 0.7
    if dtype == "bf16":
        zq, zp, zn = (synth.bf16_round(a) for a in (zq, zp, zn))
    print(f"[case] loss kernel {dtype} B={B} n_neg={n_neg} d={d}", flush=True)
    dev = lambda a: torch.as_tensor(a).to(device="cuda", dtype=torch_dtype(dtype))
    loss, per = ps.max_margin_loss(dev(zq), dev(zp), dev(zn), 0.1)
    torch.cuda.synchronize()
    ref_loss, ref_per = orc.max_margin_loss(zq, zp, zn, 0.1)
    assert 0.0 < ref_loss
    np.testing.assert_allclose(per.cpu().numpy(), ref_per, rtol=1e-5, atol=2e-6)
    assert abs(float(loss.item()) - ref_loss) <= 1e-5 * abs(ref_loss) + 2e-6


def _loss_bound(g, o, B, n_neg, valid=None):
    """Largest |loss_g - loss_o| the row errors g - o allow (see module doc);
    rows past the shared negatives are the pairs' hard negatives (pair-major),
    valid[b][j] marking the present ones."""
    dz = np.linalg.norm(g - o, axis=1)
    no = np.linalg.norm(o, axis=1)
    q, p, n = slice(0, B), slice(B, 2 * B), slice(2 * B, 2 * B + n_neg)
    dq, dp, dn = dz[q], dz[p], dz[n]
    nq, np_, nn = no[q], no[p], no[n]
    neg_sum = (dq[:, None] * nn[None, :] + nq[:, None] * dn[None, :]
               + dq[:, None] * dn[None, :]).sum(axis=1)
    count = np.full(B, float(n_neg))
    if valid is not None:
        k = valid.shape[1]
        dh = dz[2 * B + n_neg:].reshape(B, k)
        nh = no[2 * B + n_neg:].reshape(B, k)
        hard = dq[:, None] * nh + nq[:, None] * dh + dq[:, None] * dh
        neg_sum += np.where(valid, hard, 0.0).sum(axis=1)
        count += valid.sum(axis=1)
    pos_term = dq * np_ + nq * dp + dq * dp
    return float((neg_sum / count + pos_term).mean())


def _run_minibatch(orc, wl, data, idx, wts, B, n_neg, seed=0, dataflow="pool_then_dense",
                   mlp=None, hard_k=0):
    import paper_1806_01973_amd as ps
    q, p, n = synth.minibatch_pairs(wl, data["offsets"], data["col"], B, n_neg, seed=seed)
    g = ps.DeviceGraph(data["offsets"], data["col"], wl.num_pins, wl.num_boards)
    layers = [ps.DeviceLayer(L["Q"], L["q"], L["W"], L["w"], dtype=torch_dtype(wl.dtype),
                             dataflow=dataflow)
              for L in data["layers"]]
    x = torch.as_tensor(data["x"]).to(device="cuda", dtype=torch_dtype(wl.dtype))
    dmlp = None if mlp is None else ps.DeviceMLP(mlp["G1"], mlp["g"], mlp["G2"],
                                                 dtype=torch_dtype(wl.dtype))
    hard = valid = dh = None
    if hard_k:
        # Hard negatives of the queries from the oracle (Sec. 3.3), a few
        # entries knocked out to exercise absent ones.
        hard = orc.hard_negatives(data["offsets"], data["col"], wl.num_pins, wl.seed + 7, 300,
                                  3, q, 20, 200, hard_k)
        hard[1::5, 0] = -1
        valid = hard >= 0
        dh = torch.as_tensor(hard).cuda()
    mb = ps.Minibatch(g, layers, wl.walks, wl.hops, wl.T, wl.seed, B, n_neg, mlp=dmlp,
                      num_hard=hard_k)
    dq, dp, dn = (torch.as_tensor(a).cuda() for a in (q, p, n))
    mb.run(x, dq, dp, dn, 0.1, hard=dh)
    torch.cuda.synchronize()
    loss1 = mb.loss.clone()
    z = to_f64(mb.z)
    per = mb.per_pair.cpu().numpy().copy()
    sizes = mb.sizes()
    mb.run(x, dq, dp, dn, 0.1, hard=dh)  # run-to-run determinism
    torch.cuda.synchronize()
    assert torch.equal(loss1, mb.loss)
    parts = [q, p, n] + ([hard[valid]] if hard_k else [])
    targets = np.concatenate(parts).astype(np.int32)
    ref_sets = orc.minibatch_sets(targets, wl.K, idx)
    assert sizes == [len(s) for s in ref_sets], (sizes, [len(s) for s in ref_sets])
    ref_t = orc.minibatch_embed(targets, data["x"], data["layers"], idx, wts)
    if mlp is not None:
        ref_t = orc.output_mlp(ref_t, mlp["G1"], mlp["g"], mlp["G2"])
    nt = 2 * B + n_neg
    ref_z = ref_t[:nt]
    zhard = None
    if hard_k:
        zhard = np.zeros((B, hard_k, ref_t.shape[1]))
        zhard[valid] = ref_t[nt:]
        ref_z = np.concatenate([ref_z, zhard.reshape(B * hard_k, -1)])
    stats = check_embeddings(z, ref_z, wl.dtype, f"minibatch {wl.name}")
    ref_loss, ref_per = orc.max_margin_loss(ref_z[:B], ref_z[B:2 * B], ref_z[2 * B:nt], 0.1,
                                            zhard, valid)
    bound = _loss_bound(z, ref_z, B, n_neg, valid) + 1e-5
    got = float(loss1.item())
    assert abs(got - ref_loss) <= bound, (got, ref_loss, bound)
    print(f"[ok] minibatch {wl.name}: sets {sizes}, loss {got:.6f} vs {ref_loss:.6f} "
          f"(bound {bound:.2e}), {stats}", flush=True)
    return sizes


@pytest.mark.parametrize("dataflow", ["pool_then_dense", "dense_then_pool"])
def test_minibatch_tiny(orc, dataflow):
    wl = synth.WORKLOADS["tiny"]
    data = synth.make_workload(wl)
    idx, cnt, wts, _ = orc.build_neighborhoods(data["offsets"], data["col"], wl.num_pins,
                                               wl.seed, wl.walks, wl.hops, wl.T)
    print(f"[case] minibatch tiny {dataflow}", flush=True)
    _run_minibatch(orc, wl, data, idx, wts, B=64, n_neg=20, dataflow=dataflow)


@pytest.mark.parametrize("dataflow", ["pool_then_dense", "dense_then_pool"])
def test_minibatch_full(orc, medium_bundle, dataflow):
    # The minibatch-shaped workload: the 1.2M-node graph, 2,048 query pins with
    # one positive each and 500 shared negatives, bf16, dims 256 -> 512 -> 256.
    wl = synth.WORKLOADS["minibatch"]
    b = medium_bundle
    assert (wl.seed, wl.walks, wl.hops, wl.T) == (b["wl"].seed, b["wl"].walks, b["wl"].hops,
                                                 b["wl"].T)
    data = dict(b["data"])
    data["x"] = synth.make_features(wl, data["offsets"], data["col"])
    data["layers"] = synth.make_layers(wl)
    print(f"[case] minibatch full (2048 pairs, 500 negatives, bf16) {dataflow}", flush=True)
    sizes = _run_minibatch(orc, wl, data, b["idx"], b["wts"], B=2048, n_neg=500,
                           dataflow=dataflow)
    assert sizes[2] <= 2 * 2048 + 500 and sizes[1] > sizes[2] and sizes[0] > sizes[1]


@pytest.mark.parametrize("dataflow", ["pool_then_dense", "dense_then_pool"])
def test_minibatch_with_output_layers(orc, dataflow):
    # Algorithm 2 in full: the K layers, then z = G2 ReLU(G1 h + g), and the
    # loss of Eq. 1 on z.
    wl = synth.WORKLOADS["tiny"]
    data = synth.make_workload(wl)
    idx, cnt, wts, _ = orc.build_neighborhoods(data["offsets"], data["col"], wl.num_pins,
                                               wl.seed, wl.walks, wl.hops, wl.T)
    mlp = synth.make_mlp(wl.d_out, 96, 48, seed=17)
    print(f"[case] minibatch tiny with output layers {dataflow}", flush=True)
    _run_minibatch(orc, wl, data, idx, wts, B=64, n_neg=20, dataflow=dataflow, mlp=mlp)


@pytest.mark.parametrize("dataflow", ["pool_then_dense", "dense_then_pool"])
def test_minibatch_with_hard_negatives(orc, dataflow):
    # Sec. 3.3: each query's hard negatives join the targets of Algorithm 2 and
    # the query's negative set in Eq. 1.
    wl = synth.WORKLOADS["tiny"]
    data = synth.make_workload(wl)
    idx, cnt, wts, _ = orc.build_neighborhoods(data["offsets"], data["col"], wl.num_pins,
                                               wl.seed, wl.walks, wl.hops, wl.T)
    print(f"[case] minibatch tiny with hard negatives {dataflow}", flush=True)
    _run_minibatch(orc, wl, data, idx, wts, B=64, n_neg=20, dataflow=dataflow, hard_k=3)


def test_minibatch_full_with_hard_negatives(orc, medium_bundle):
    wl = synth.WORKLOADS["minibatch"]
    b = medium_bundle
    data = dict(b["data"])
    data["x"] = synth.make_features(wl, data["offsets"], data["col"])
    data["layers"] = synth.make_layers(wl)
    print("[case] minibatch full with 2 hard negatives per pair", flush=True)
    sizes = _run_minibatch(orc, wl, data, b["idx"], b["wts"], B=2048, n_neg=500,
                           dataflow="dense_then_pool", hard_k=2)
    assert sizes[2] <= 4 * 2048 + 500


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("B,n_neg,k,d", [(333, 77, 5, 200), (64, 500, 1, 256), (19, 45, 40, 1024),
                                         (5, 3, 2, 13)])
def test_loss_kernel_with_hard_negatives(orc, dtype, B, n_neg, k, d):
    import paper_1806_01973_amd as ps
    rng = np.random.default_rng(5)
    zq, zp, zn = _unit_rows(rng, B, d), _unit_rows(rng, B, d), _unit_rows(rng, n_neg, d)
    zh = _unit_rows(rng, B * k, d).reshape(B, k, d)
    zh[: B // 2] = 0.5 * zh[: B // 2] + 0.5 * zq[: B // 2, None, :]  # hard: close to the query
    zp[: B // 3] = zq[: B // 3] * 0.3 + zp[: B // 3] * 0.7
    if dtype == "bf16":
        zq, zp, zn, zh = (synth.bf16_round(a) for a in (zq, zp, zn, zh))
    print(f"[case] loss kernel with hard negatives {dtype} B={B} n_neg={n_neg} k={k} d={d}",
          flush=True)
    dev = lambda a: torch.as_tensor(np.ascontiguousarray(a)).to(device="cuda",
                                                               dtype=torch_dtype(dtype))
    loss, per = ps.max_margin_loss(dev(zq), dev(zp), dev(zn), 0.1, zhard=dev(zh))
    torch.cuda.synchronize()
    ref_loss, ref_per = orc.max_margin_loss(zq, zp, zn, 0.1, zh)
    _, shared_only = orc.max_margin_loss(zq, zp, zn, 0.1)
    assert not np.allclose(ref_per, shared_only)  # the hard terms matter
    np.testing.assert_allclose(per.cpu().numpy(), ref_per, rtol=1e-5, atol=2e-6)
    assert abs(float(loss.item()) - ref_loss) <= 1e-5 * abs(ref_loss) + 2e-6
