"""C-ABI checks that need no GPU: the library loads, exports every entry point
include/pinsage.h declares, and rejects malformed arguments on the host before
any HIP call (the pointers passed here are never dereferenced)."""

import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "pinsage.h")


@pytest.fixture(scope="module")
def L():
    from paper_1806_01973_amd import _lib
    if not os.path.exists(_lib.LIB_PATH):
        pytest.skip("libpinsage.so not built (run __graft_entry__.build())")
    _lib.lib()
    return _lib


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(pinsage_[a-z_0-9]+)\s*\(", text)))


def test_exports_every_declared_symbol(L):
    names = _declared()
    assert len(names) >= 10
    for n in names:
        assert hasattr(L.lib(), n), n
    assert sorted(L.EXPORTED) == names


def test_version_and_status_strings(L):
    lib = L.lib()
    assert lib.pinsage_version() == 12
    for code in (0, -1, -2, -3, -4):
        assert lib.pinsage_status_string(code)
    assert lib.pinsage_status_string(-99) == b"unknown status"


FAKE = 0x10000  # never dereferenced: every call below fails validation first


def _graph(L, **kw):
    g = dict(num_pins=10, num_boards=5, nnz=40, offset_type=L.PINSAGE_I32, row_offsets=FAKE,
             col=FAKE)
    g.update(kw)
    return L.Graph(**g)


def _layer(L, **kw):
    d = dict(d_in=64, m=128, d_out=64, dtype=L.PINSAGE_F32, Q=FAKE, q=FAKE, W=FAKE, w=FAKE)
    d.update(kw)
    return L.Layer(**d)


def test_build_neighborhoods_validation(L):
    lib = L.lib()
    walk = L.WalkParams(1, 10, 2, 8)
    nb = L.Neighborhoods(15, 8, FAKE, FAKE, None)
    call = lambda g, w, src, ns, n: lib.pinsage_build_neighborhoods(
        ctypes.byref(g) if g is not None else None, ctypes.byref(w) if w is not None else None,
        src, ns, ctypes.byref(n) if n is not None else None, None, None)
    assert call(None, walk, None, 15, nb) == L.PINSAGE_EINVAL
    assert call(_graph(L), None, None, 15, nb) == L.PINSAGE_EINVAL
    assert call(_graph(L), walk, None, 14, nb) == L.PINSAGE_EINVAL  # NULL sources needs all nodes
    assert b"num_sources" in lib.pinsage_last_error()
    assert call(_graph(L, num_pins=-1), walk, None, 15, nb) == L.PINSAGE_EINVAL
    assert call(_graph(L, nnz=2**31), walk, None, 15, nb) == L.PINSAGE_EUNSUPPORTED
    assert call(_graph(L, offset_type=7), walk, None, 15, nb) == L.PINSAGE_EINVAL
    assert call(_graph(L, num_pins=2**31), walk, None, 15, nb) == L.PINSAGE_EUNSUPPORTED
    assert call(_graph(L), L.WalkParams(1, 600, 2, 8), None, 15, nb) == L.PINSAGE_EUNSUPPORTED
    assert call(_graph(L), L.WalkParams(1, 0, 2, 8), None, 15, nb) == L.PINSAGE_EINVAL
    assert call(_graph(L), L.WalkParams(1, 10, 2, 257), None, 15, nb) == L.PINSAGE_EUNSUPPORTED
    assert call(_graph(L), walk, None, 15, L.Neighborhoods(15, 9, FAKE, FAKE, None)) == \
        L.PINSAGE_EINVAL  # top_t mismatch
    assert call(_graph(L), walk, None, 15, L.Neighborhoods(14, 8, FAKE, FAKE, None)) == \
        L.PINSAGE_EINVAL  # row mismatch
    assert call(_graph(L), walk, None, 15, L.Neighborhoods(15, 8, None, FAKE, None)) == \
        L.PINSAGE_EINVAL


def test_walk_table_validation(L):
    lib = L.lib()
    n = ctypes.c_size_t(7)
    assert lib.pinsage_walk_table_size(ctypes.byref(_graph(L)), ctypes.byref(n)) == L.PINSAGE_OK
    assert n.value == 40 * 16
    assert lib.pinsage_walk_table_size(ctypes.byref(_graph(L)), None) == L.PINSAGE_EINVAL
    g64 = _graph(L, nnz=2**31, offset_type=L.PINSAGE_I64)
    assert lib.pinsage_walk_table_size(ctypes.byref(g64), ctypes.byref(n)) == L.PINSAGE_EUNSUPPORTED
    assert n.value == 0
    assert lib.pinsage_walk_table_size(ctypes.byref(_graph(L, num_pins=-1)),
                                       ctypes.byref(n)) == L.PINSAGE_EINVAL
    build = lambda g, t, b: lib.pinsage_build_walk_table(ctypes.byref(g), t, b, None)
    assert build(_graph(L), FAKE, 40 * 16 - 1) == L.PINSAGE_EWORKSPACE
    assert build(_graph(L), None, 40 * 16) == L.PINSAGE_EINVAL
    assert build(_graph(L), FAKE + 8, 40 * 16) == L.PINSAGE_EINVAL  # alignment
    assert build(g64, FAKE, 2**36) == L.PINSAGE_EUNSUPPORTED
    # A graph carrying a walk table: checked wherever the graph is.
    walk = L.WalkParams(1, 10, 2, 8)
    nb = L.Neighborhoods(15, 8, FAKE, FAKE, None)
    for g, want in ((_graph(L, walk_table=FAKE + 4), L.PINSAGE_EINVAL),
                    (_graph(L, nnz=2**31, offset_type=L.PINSAGE_I64, walk_table=FAKE),
                     L.PINSAGE_EUNSUPPORTED)):
        assert lib.pinsage_build_neighborhoods(ctypes.byref(g), ctypes.byref(walk), None, 15,
                                               ctypes.byref(nb), None, None) == want
        assert b"walk" in lib.pinsage_last_error() or b"nnz" in lib.pinsage_last_error()


def test_hard_negatives_validation(L):
    lib = L.lib()
    hp = lambda **kw: L.HardNegativeParams(**{**dict(seed=1, walks=4096, hops=4, rank_lo=1999,
                                                      rank_hi=5000, num_per_query=3), **kw})
    call = lambda g, p, q, n, out, ws=None, wsb=0: lib.pinsage_hard_negatives(
        ctypes.byref(g) if g is not None else None, ctypes.byref(p) if p is not None else None,
        q, n, out, None, ws, wsb, None)
    assert call(None, hp(), FAKE, 4, FAKE) == L.PINSAGE_EINVAL
    assert call(_graph(L), None, FAKE, 4, FAKE) == L.PINSAGE_EINVAL
    assert call(_graph(L), hp(walks=0), FAKE, 4, FAKE) == L.PINSAGE_EINVAL
    assert call(_graph(L), hp(walks=1 << 21, hops=3), FAKE, 4, FAKE) == L.PINSAGE_EUNSUPPORTED
    assert b"exceeds" in lib.pinsage_last_error()
    # Budgets past the on-chip slots count visits in the workspace, and rank
    # only up to rank_hi = 8192 there.
    n = ctypes.c_size_t(1)
    assert lib.pinsage_hard_negatives_workspace_size(ctypes.byref(hp()), 4, ctypes.byref(n)) == 0
    assert n.value == 0  # 16384 landings: on chip
    big = hp(hops=5)     # 20480 landings: 3 partitions' buckets of 12288, overflow
    per = 4 * (3 * 12288 + 4 * 20480)  # list twice, (pin, count) list
    assert per % 256 == 0
    assert lib.pinsage_hard_negatives_workspace_size(ctypes.byref(big), 4, ctypes.byref(n)) == 0
    assert n.value == 4 * per
    assert lib.pinsage_hard_negatives_workspace_size(ctypes.byref(big), 10_000,
                                                     ctypes.byref(n)) == 0
    assert n.value == 256 * per  # at most 256 resident workgroups
    assert call(_graph(L), big, FAKE, 4, FAKE) == L.PINSAGE_EWORKSPACE
    assert call(_graph(L), big, FAKE, 4, FAKE, FAKE, 100) == L.PINSAGE_EWORKSPACE
    assert call(_graph(L), big, FAKE, 4, FAKE, FAKE + 8, 1 << 30) == L.PINSAGE_EINVAL
    assert call(_graph(L), hp(hops=5, rank_hi=8193), FAKE, 4, FAKE, FAKE, 1 << 30) == \
        L.PINSAGE_EUNSUPPORTED
    assert b"8192" in lib.pinsage_last_error()
    assert call(_graph(L), hp(rank_lo=-1), FAKE, 4, FAKE) == L.PINSAGE_EINVAL
    assert call(_graph(L), hp(rank_lo=10, rank_hi=10), FAKE, 4, FAKE) == L.PINSAGE_EINVAL
    assert call(_graph(L), hp(num_per_query=-1), FAKE, 4, FAKE) == L.PINSAGE_EINVAL
    assert call(_graph(L), hp(), None, 4, FAKE) == L.PINSAGE_EINVAL
    assert call(_graph(L), hp(), FAKE, 4, None) == L.PINSAGE_EINVAL
    assert call(_graph(L), hp(), FAKE, -1, FAKE) == L.PINSAGE_EINVAL
    assert call(_graph(L, offset_type=7), hp(), FAKE, 4, FAKE) == L.PINSAGE_EINVAL
    # Nothing to do: accepted without touching the device.
    assert call(_graph(L), hp(), None, 0, None) == L.PINSAGE_OK
    assert call(_graph(L), hp(num_per_query=0), FAKE, 4, None) == L.PINSAGE_OK


def test_graph_neighborhoods_and_bipartite_validation(L):
    lib = L.lib()
    nb = L.Neighborhoods(15, 8, FAKE, FAKE, None)
    call = lambda g, src, ns, n: lib.pinsage_build_graph_neighborhoods(
        ctypes.byref(g) if g is not None else None, 3, src, ns,
        ctypes.byref(n) if n is not None else None, None)
    assert call(None, None, 15, nb) == L.PINSAGE_EINVAL
    assert call(_graph(L), None, 14, nb) == L.PINSAGE_EINVAL
    assert call(_graph(L), None, 15, None) == L.PINSAGE_EINVAL
    assert call(_graph(L), None, 15, L.Neighborhoods(15, 257, FAKE, FAKE, None)) == \
        L.PINSAGE_EUNSUPPORTED
    assert call(_graph(L), FAKE, 3, L.Neighborhoods(4, 8, FAKE, FAKE, None)) == L.PINSAGE_EINVAL
    n = ctypes.c_size_t(0)
    g = _graph(L)
    layers = (L.Layer * 3)(_layer(L), _layer(L), _layer(L))
    ws = lib.pinsage_embed_all_bipartite_workspace_size
    assert ws(ctypes.byref(g), layers, 2, ctypes.byref(n)) == 0
    a = lambda b: (b + 255) // 256 * 256
    # Every node projected: P (15 x 128) and the pooled chunk (15 x 128) fp32,
    # one h buffer (15 x 64) and the pin row map (15 int32).
    assert n.value == a(15 * 128 * 4) + a(15 * 128 * 4) + a(15 * 64 * 4) + a(15 * 4)
    assert ws(ctypes.byref(g), layers, 3, ctypes.byref(n)) == L.PINSAGE_EUNSUPPORTED  # odd K
    assert b"even" in lib.pinsage_last_error()
    assert ws(ctypes.byref(g), layers, 0, ctypes.byref(n)) == L.PINSAGE_EINVAL
    nb15 = L.Neighborhoods(15, 8, FAKE, FAKE, None)
    st = lib.pinsage_embed_all_bipartite(ctypes.byref(g), 1, layers, 2, FAKE, ctypes.byref(nb15),
                                         FAKE, FAKE, 16, None)
    assert st == L.PINSAGE_EWORKSPACE
    st = lib.pinsage_embed_all_bipartite(ctypes.byref(g), 1, layers, 2, None, ctypes.byref(nb15),
                                         FAKE, FAKE, 1 << 30, None)
    assert st == L.PINSAGE_EINVAL


def test_layer_validation_and_workspace_sizes(L):
    lib = L.lib()
    n = ctypes.c_size_t(0)
    ly = _layer(L)
    assert lib.pinsage_convolve_workspace_size(ctypes.byref(ly), 100, 300, ctypes.byref(n)) == 0
    # P (100 x 128 fp32) + pooled rows (300 x 128 fp32), each 256-aligned.
    assert n.value == 51200 + 153600
    lyb = _layer(L, dtype=L.PINSAGE_BF16)
    assert lib.pinsage_convolve_workspace_size(ctypes.byref(lyb), 100, 300, ctypes.byref(n)) == 0
    assert n.value == 25600 + 76800
    # Dense then pool: R (100 x 64 fp32) + P chunk (100 x 128) + pooled rows (300 x 64).
    lyd = _layer(L, dataflow=L.PINSAGE_DENSE_THEN_POOL)
    assert lib.pinsage_convolve_workspace_size(ctypes.byref(lyd), 100, 300, ctypes.byref(n)) == 0
    assert n.value == 25600 + 51200 + 76800
    for bad, code in [(dict(d_in=60), L.PINSAGE_EUNSUPPORTED), (dict(d_out=1024), L.PINSAGE_EUNSUPPORTED),
                      (dict(m=0), L.PINSAGE_EINVAL), (dict(Q=None), L.PINSAGE_EINVAL),
                      (dict(dtype=5), L.PINSAGE_EINVAL), (dict(dataflow=2), L.PINSAGE_EINVAL),
                      (dict(pool=3), L.PINSAGE_EINVAL),
                      (dict(pool=2, dataflow=1), L.PINSAGE_EUNSUPPORTED)]:
        b = _layer(L, **bad)
        assert lib.pinsage_convolve_workspace_size(ctypes.byref(b), 1, 1, ctypes.byref(n)) == code
    # Workspace too small: rejected before any launch.
    nb = L.Neighborhoods(300, 8, FAKE, FAKE, None)
    st = lib.pinsage_convolve_layer(ctypes.byref(ly), FAKE, 300, 100, None, ctypes.byref(nb), None,
                                    FAKE, 300, FAKE, 1024, None)
    assert st == L.PINSAGE_EWORKSPACE
    st = lib.pinsage_convolve_layer(ctypes.byref(ly), FAKE, 300, 400, None, ctypes.byref(nb), None,
                                    FAKE, 300, FAKE, 1 << 30, None)
    assert st == L.PINSAGE_EINVAL  # n_transform > n_in
    st = lib.pinsage_convolve_layer(ctypes.byref(ly), FAKE, 300, 100, None, ctypes.byref(nb), None,
                                    FAKE, 300, FAKE + 8, 1 << 30, None)
    assert st == L.PINSAGE_EINVAL  # misaligned workspace
    # embed_all: sizes, layer chaining, dtype consistency.
    g = _graph(L)
    layers = (L.Layer * 2)(_layer(L), _layer(L, d_in=64))
    assert lib.pinsage_embed_all_workspace_size(ctypes.byref(g), layers, 2, ctypes.byref(n)) == 0
    conv = 5120 + 7680  # P: 10 pins x 128 x 4; pooled: 15 x 128 x 4 (256-aligned)
    hbuf = 3840         # h^(1): 15 x 64 x 4
    assert n.value == conv + hbuf
    bad = (L.Layer * 2)(_layer(L), _layer(L, d_in=128))
    walk = L.WalkParams(1, 10, 2, 8)
    nbr = L.Neighborhoods(15, 8, FAKE, FAKE, None)
    st = lib.pinsage_embed_all(ctypes.byref(g), ctypes.byref(walk), bad, 2, FAKE,
                               ctypes.byref(nbr), FAKE, None, FAKE, 1 << 30, None, None)
    assert st == L.PINSAGE_EINVAL and b"d_in" in lib.pinsage_last_error()
    mixed = (L.Layer * 2)(_layer(L), _layer(L, dtype=L.PINSAGE_BF16))
    st = lib.pinsage_embed_all(ctypes.byref(g), ctypes.byref(walk), mixed, 2, FAKE,
                               ctypes.byref(nbr), FAKE, None, FAKE, 1 << 30, None, None)
    assert st == L.PINSAGE_EINVAL
    st = lib.pinsage_embed_all(ctypes.byref(g), ctypes.byref(walk), layers, 2, FAKE,
                               ctypes.byref(nbr), FAKE, None, FAKE, 64, None, None)
    assert st == L.PINSAGE_EWORKSPACE


def test_profile_read_validation(L):
    lib = L.lib()
    n = ctypes.c_int64(0)
    ms = ctypes.c_double(0)
    assert lib.pinsage_profile_read(99, ctypes.byref(n), ctypes.byref(ms)) == L.PINSAGE_EINVAL
    assert lib.pinsage_profile_enable(0) == 0
    assert lib.pinsage_profile_read(0, ctypes.byref(n), ctypes.byref(ms)) == 0
    assert n.value == 0 and ms.value == 0.0


def test_random_read_calibration_validation(L):
    lib = L.lib()
    E = L.PINSAGE_EINVAL
    f = lib.pinsage_profile_random_reads
    assert f(None, 1 << 20, 4, 8, FAKE, 256, None) == E
    assert f(FAKE, 1 << 20, 4, 8, None, 256, None) == E
    for eb in (0, 2, 12, 32):
        assert f(FAKE, 1 << 20, eb, 8, FAKE, 256, None) == E
    assert f(FAKE, 8, 16, 8, FAKE, 256, None) == E  # smaller than one element
    assert f(FAKE, 1 << 20, 16, 0, FAKE, 256, None) == E
    assert f(FAKE, 1 << 20, 16, 8, FAKE, 0, None) == E
    assert f(FAKE, 1 << 20, 12, 8, FAKE, 256, None) == E
    assert b"element size 12" in lib.pinsage_last_error()


def test_random_gather_calibration_validation(L):
    lib = L.lib()
    E = L.PINSAGE_EINVAL
    f = lib.pinsage_profile_random_gathers
    assert f(None, 1 << 20, 512, 8, 50, 1, FAKE, None) == E
    assert f(FAKE, 1 << 20, 512, 8, 50, 1, None, None) == E
    for rb in (0, 256, 768, 2048):
        assert f(FAKE, 1 << 20, rb, 8, 50, 1, FAKE, None) == E
    assert b"row size 2048" in lib.pinsage_last_error()
    assert f(FAKE + 8, 1 << 20, 512, 8, 50, 1, FAKE, None) == E  # misaligned
    assert f(FAKE, 511, 512, 8, 50, 1, FAKE, None) == E  # smaller than one row
    assert f(FAKE, 1 << 20, 512, 0, 50, 1, FAKE, None) == E
    assert f(FAKE, 1 << 20, 512, 8, 0, 1, FAKE, None) == E
    assert f(FAKE, 1 << 20, 512, 8, 65, 1, FAKE, None) == E
    assert f(FAKE, 1 << 20, 1024, 8, 33, 1, FAKE, None) == E
    assert f(FAKE, 512 << 32, 512, 8, 8, 1, FAKE, None) == L.PINSAGE_EUNSUPPORTED  # 2^32 rows


def test_minibatch_validation_and_workspace(L):
    lib = L.lib()
    n = ctypes.c_size_t(0)
    g = _graph(L)  # 15 nodes
    walk = L.WalkParams(1, 10, 2, 4)
    layers = (L.Layer * 2)(_layer(L), _layer(L))
    assert lib.pinsage_minibatch_workspace_size(ctypes.byref(g), ctypes.byref(walk), layers, 2,
                                                None, 3, 2, 0, ctypes.byref(n)) == 0
    # Frontier capacities: U2 = min(15, 2*3+2) = 8, U1 = U0 = 15 (capped by N).
    a = lambda b: (b + 255) // 256 * 256
    U = [15, 15, 8]
    want = a(15) + a(60) + a(4) + a(64) + sum(a(u * 4) for u in U)
    for k in (1, 2):
        want += a(U[k] * 4 * 4) + a(U[k] * 4 * 2) + a(U[k] * 4 * 4) + a(U[k] * 4) + a(U[k] * 64 * 4)
    want += a(8 * 4) + a(3 * 4)
    conv = max(a(U[k - 1] * 128 * 4) + a(U[k] * 128 * 4) for k in (1, 2))
    want += a(conv)
    assert n.value == want
    assert lib.pinsage_minibatch_workspace_size(ctypes.byref(g), ctypes.byref(walk), layers, 2,
                                                None, 0, 2, 0, ctypes.byref(n)) == L.PINSAGE_EINVAL
    assert lib.pinsage_minibatch_workspace_size(ctypes.byref(g), ctypes.byref(walk), layers, 9,
                                                None, 3, 2, 0, ctypes.byref(n)) == L.PINSAGE_EUNSUPPORTED
    assert lib.pinsage_minibatch_workspace_size(ctypes.byref(g), ctypes.byref(walk), layers, 2,
                                                None, 3, 2, -1, ctypes.byref(n)) == L.PINSAGE_EINVAL
    # Hard negatives widen the level-K capacity: U2 = min(15, 2*3+2+3*2) = 14,
    # and the target row table to 14 entries.
    n_h = ctypes.c_size_t(0)
    assert lib.pinsage_minibatch_workspace_size(ctypes.byref(g), ctypes.byref(walk), layers, 2,
                                                None, 3, 2, 2, ctypes.byref(n_h)) == 0
    Uh = [15, 15, 14]
    want_h = a(15) + a(60) + a(4) + a(64) + sum(a(u * 4) for u in Uh)
    for k in (1, 2):
        want_h += (a(Uh[k] * 4 * 4) + a(Uh[k] * 4 * 2) + a(Uh[k] * 4 * 4) + a(Uh[k] * 4) +
                   a(Uh[k] * 64 * 4))
    want_h += a(14 * 4) + a(3 * 4)
    want_h += a(max(a(Uh[k - 1] * 128 * 4) + a(Uh[k] * 128 * 4) for k in (1, 2)))
    assert n_h.value == want_h
    pairs = L.Pairs(3, 2, FAKE, None, FAKE, 0.1, 0, None)
    st = lib.pinsage_minibatch_forward(ctypes.byref(g), ctypes.byref(walk), layers, 2, None, FAKE,
                                       ctypes.byref(pairs), FAKE, None, None, None, None, FAKE,
                                       1 << 30, None)
    assert st == L.PINSAGE_EINVAL
    pairs = L.Pairs(3, 2, FAKE, FAKE, FAKE, 0.1, 0, None)
    st = lib.pinsage_minibatch_forward(ctypes.byref(g), ctypes.byref(walk), layers, 2, None, FAKE,
                                       ctypes.byref(pairs), FAKE, None, None, None, None, FAKE, 16,
                                       None)
    assert st == L.PINSAGE_EWORKSPACE
    pairs = L.Pairs(3, 2, FAKE, FAKE, FAKE, 0.1, 2, None)  # hard negatives missing
    st = lib.pinsage_minibatch_forward(ctypes.byref(g), ctypes.byref(walk), layers, 2, None, FAKE,
                                       ctypes.byref(pairs), FAKE, None, None, None, None, FAKE,
                                       1 << 30, None)
    assert st == L.PINSAGE_EINVAL
    # Standalone loss: per_pair is required, d is bounded.
    st = lib.pinsage_max_margin_loss(FAKE, FAKE, 4, FAKE, 5, None, 0, 64, L.PINSAGE_F32, 0.1,
                                     FAKE, None, None)
    assert st == L.PINSAGE_EINVAL
    st = lib.pinsage_max_margin_loss(FAKE, FAKE, 4, FAKE, 5, None, 0, 2048, L.PINSAGE_F32, 0.1,
                                     FAKE, FAKE, None)
    assert st == L.PINSAGE_EUNSUPPORTED
    st = lib.pinsage_max_margin_loss(FAKE, FAKE, 4, FAKE, 5, None, 3, 64, L.PINSAGE_F32, 0.1,
                                     FAKE, FAKE, None)
    assert st == L.PINSAGE_EINVAL  # zhard missing
    st = lib.pinsage_max_margin_loss(FAKE, FAKE, 4, FAKE, 5, FAKE, -1, 64, L.PINSAGE_F32, 0.1,
                                     FAKE, FAKE, None)
    assert st == L.PINSAGE_EINVAL


def _mlp(L, **kw):
    d = dict(d_in=64, d_hidden=96, d_out=32, dtype=L.PINSAGE_F32, G1=FAKE, g=FAKE, G2=FAKE)
    d.update(kw)
    return L.MLP(**d)


def test_output_mlp_validation(L):
    lib = L.lib()
    n = ctypes.c_size_t(0)
    m = _mlp(L)
    assert lib.pinsage_output_mlp_workspace_size(ctypes.byref(m), 300, ctypes.byref(n)) == 0
    assert n.value == 300 * 96 * 4 // 256 * 256 + (256 if 300 * 96 * 4 % 256 else 0)
    for bad, code in [(dict(d_in=60), L.PINSAGE_EUNSUPPORTED), (dict(d_hidden=0), L.PINSAGE_EINVAL),
                      (dict(G2=None), L.PINSAGE_EINVAL), (dict(dtype=9), L.PINSAGE_EINVAL),
                      (dict(d_out=16384), L.PINSAGE_EUNSUPPORTED)]:
        b = _mlp(L, **bad)
        assert lib.pinsage_output_mlp_workspace_size(ctypes.byref(b), 1, ctypes.byref(n)) == code
    assert lib.pinsage_output_mlp(ctypes.byref(m), FAKE, 300, FAKE, FAKE, 1024, None) == \
        L.PINSAGE_EWORKSPACE
    assert lib.pinsage_output_mlp(ctypes.byref(m), FAKE, 300, FAKE, FAKE + 8, 1 << 30, None) == \
        L.PINSAGE_EINVAL
    assert lib.pinsage_output_mlp(ctypes.byref(m), FAKE, 0, FAKE, None, 0, None) == 0
    # Minibatch with output layers: d_in must match the last layer, dtype must match.
    g = _graph(L)
    walk = L.WalkParams(1, 10, 2, 4)
    layers = (L.Layer * 2)(_layer(L), _layer(L))
    bad = _mlp(L, d_in=32)
    assert lib.pinsage_minibatch_workspace_size(ctypes.byref(g), ctypes.byref(walk), layers, 2,
                                                ctypes.byref(bad), 3, 2, 0, ctypes.byref(n)) == \
        L.PINSAGE_EINVAL
    ok = _mlp(L, d_in=64)
    n0 = ctypes.c_size_t(0)
    assert lib.pinsage_minibatch_workspace_size(ctypes.byref(g), ctypes.byref(walk), layers, 2,
                                                None, 3, 2, 0, ctypes.byref(n0)) == 0
    assert lib.pinsage_minibatch_workspace_size(ctypes.byref(g), ctypes.byref(walk), layers, 2,
                                                ctypes.byref(ok), 3, 2, 0, ctypes.byref(n)) == 0
    a = lambda b: (b + 255) // 256 * 256
    assert n.value == n0.value + a(8 * 32 * 4) + a(8 * 96 * 4)  # z and hidden rows of S^(2)


def test_schedule_validation(L):
    # Host-only paths: the share and the output pointer are checked before any
    # device call; destroying NULL is a no-op.
    lib = L.lib()
    h = ctypes.c_void_p(None)
    for bad in (8, 0, -1):
        assert lib.pinsage_schedule_create(bad, ctypes.byref(h)) == L.PINSAGE_EINVAL
        assert b"cu_eighths" in lib.pinsage_last_error()
        assert h.value is None
    assert lib.pinsage_schedule_create(4, None) == L.PINSAGE_EINVAL
    assert lib.pinsage_schedule_destroy(None) == 0
