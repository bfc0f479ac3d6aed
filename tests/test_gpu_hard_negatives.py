"""GPU parity: hard negative items (Sec. 3.3) must equal the oracle's draws
bit for bit (they are node ids), and the edge-step total must equal the sum of
the oracle's per-query walk steps.

Covers every visit-slot width of the kernel (walks * hops up to 1024 * E for
E = 1 .. 16), the 1.2M-node graph at the hard negative workload (4096 walks of
4 landings, the paper's rank window 2000-5000, a ragged query count over many
workgroups), windows past the ranked pins, boards, invalid and repeated query
ids, int64 row offsets and num_per_query = 0.
"""

import numpy as np
import pytest
import torch

import synth

pytestmark = pytest.mark.gpu


def _gpu(off, col, P, B, queries, k, seed, walks, hops, lo, hi, offsets64=None):
    import paper_1806_01973_amd as ps
    g = ps.DeviceGraph(off, col, P, B, offsets64=offsets64)
    q = torch.as_tensor(np.asarray(queries, np.int32)).cuda()
    out, steps = ps.hard_negatives(g, q, k, seed, walks, hops, lo, hi, count_steps=True)
    torch.cuda.synchronize()
    return out.cpu().numpy(), int(steps.item())


@pytest.fixture(scope="module")
def tiny():
    wl = synth.WORKLOADS["tiny"]
    off, col, _ = synth.make_graph(wl)
    return wl, off, col


def _queries(wl, n, seed):
    rng = np.random.default_rng(seed)
    N = wl.num_pins + wl.num_boards
    q = rng.integers(0, N, n).astype(np.int32)
    q[::7] = rng.integers(0, wl.num_pins, len(q[::7]))  # mostly pins, some boards
    return q


@pytest.mark.parametrize("walks,hops,lo,hi,k", [
    (200, 3, 20, 60, 5),        # 600 slots: one per thread
    (1000, 2, 0, 10, 3),        # 2000 slots
    (1024, 4, 100, 400, 17),    # 4096
    (4096, 2, 300, 1200, 2),    # 8192
    (4096, 4, 1999, 5000, 4),   # 16384, the paper's window (beyond a 2000-pin graph)
    (16384, 1, 500, 501, 9),    # one-rank window, single-landing walks
])
def test_tiny_widths(orc, tiny, walks, hops, lo, hi, k):
    wl, off, col = tiny
    q = _queries(wl, 300, walks + hops)
    print(f"[case] tiny hard negatives W={walks} H={hops} [{lo},{hi}) k={k}", flush=True)
    got, steps = _gpu(off, col, wl.num_pins, wl.num_boards, q, k, 13, walks, hops, lo, hi)
    ref = orc.hard_negatives(off, col, wl.num_pins, 13, walks, hops, q, lo, hi, k)
    np.testing.assert_array_equal(got, ref)
    want = sum(orc.walk_visits(off, col, wl.num_pins, 13, u, walks, hops)[1] for u in q.tolist())
    assert steps == want


def test_degenerate_queries(orc):
    P, B = 3, 2
    off, col = synth.csr_from_edges(P, B, [(0, 0), (1, 0)])  # pin 2, board 1 isolated
    q = np.array([0, 2, 4, -1, 5, 1, 0, 2**31 - 1], np.int32)
    print("[case] hard negatives on isolated / invalid queries", flush=True)
    for lo, hi in [(0, 5), (1, 5), (0, 1)]:
        got, _ = _gpu(off, col, P, B, q, 3, 1, 10, 2, lo, hi)
        np.testing.assert_array_equal(got, orc.hard_negatives(off, col, P, 1, 10, 2, q, lo, hi, 3))
    got, steps = _gpu(off, col, P, B, q, 0, 1, 10, 2, 0, 5)
    assert got.shape == (len(q), 0)
    # Pins 0, 1, 0 walk 10 times with 4 edge steps each; the other queries are
    # isolated (pin 2, board 4) or outside the graph.
    assert steps == 3 * 10 * 4


def test_int64_offsets_and_repeats(orc, tiny):
    wl, off, col = tiny
    q = np.repeat(_queries(wl, 40, 3), 3)
    print("[case] hard negatives int64 offsets, repeated queries", flush=True)
    got, _ = _gpu(off, col, wl.num_pins, wl.num_boards, q, 6, 21, 512, 3, 10, 90, offsets64=True)
    ref = orc.hard_negatives(off, col, wl.num_pins, 21, 512, 3, q, 10, 90, 6)
    np.testing.assert_array_equal(got, ref)
    np.testing.assert_array_equal(got[0::3], got[1::3])


def test_medium_workload(orc):
    wl = synth.WORKLOADS["medium"]
    off, col, _ = synth.make_graph(wl)
    rng = np.random.default_rng(8)
    q = rng.integers(0, wl.num_pins, 1000).astype(np.int32)
    walks, hops, lo, hi, k = 4096, 4, 1999, 5000, 8
    print(f"[case] medium hard negatives n={len(q)} W={walks} H={hops} [{lo},{hi}) k={k}",
          flush=True)
    got, _ = _gpu(off, col, wl.num_pins, wl.num_boards, q, k, 99, walks, hops, lo, hi)
    ref = orc.hard_negatives(off, col, wl.num_pins, 99, walks, hops, q, lo, hi, k)
    np.testing.assert_array_equal(got, ref)
    assert np.all(got < wl.num_pins)
    assert (got >= 0).mean() > 0.9  # most queries reach past rank 5000


def test_more_queries_than_workgroups(orc, tiny):
    # 9,000 queries: past the 8,192-workgroup grid, so workgroups take a second
    # query (grid-stride), with the one-slot-per-thread width.
    wl, off, col = tiny
    rng = np.random.default_rng(12)
    q = rng.integers(-5, wl.num_nodes + 5, 9000).astype(np.int32)
    print("[case] hard negatives, 9000 queries (grid-stride)", flush=True)
    got, steps = _gpu(off, col, wl.num_pins, wl.num_boards, q, 3, 31, 100, 2, 5, 40)
    np.testing.assert_array_equal(got, orc.hard_negatives(off, col, wl.num_pins, 31, 100, 2, q,
                                                          5, 40, 3))
    valid = [int(u) for u in q if 0 <= u < wl.num_nodes]
    assert steps == sum(orc.walk_visits(off, col, wl.num_pins, 31, u, 100, 2)[1] for u in valid)


# ---- walk budgets past the 16,384 on-chip slots: visits counted in a global
# table of the workspace, ranks selected by count threshold and id -----------

def test_global_table_medium_paper_window(orc):
    # 131,072 landings per query on the 1.2M-node graph: the paper's window
    # [1999, 5000) is then decided by visit counts (pins visited once rank
    # last), not by the id order of single visits.
    wl = synth.WORKLOADS["medium"]
    off, col, _ = synth.make_graph(wl)
    rng = np.random.default_rng(9)
    q = rng.integers(0, wl.num_pins, 400).astype(np.int32)
    walks, hops, lo, hi, k = 32768, 4, 1999, 5000, 8
    print(f"[case] medium hard negatives, global table n={len(q)} W={walks} H={hops} "
          f"[{lo},{hi}) k={k}", flush=True)
    got, steps = _gpu(off, col, wl.num_pins, wl.num_boards, q, k, 77, walks, hops, lo, hi)
    ref = orc.hard_negatives(off, col, wl.num_pins, 77, walks, hops, q, lo, hi, k)
    np.testing.assert_array_equal(got, ref)
    # The window is inside the repeated-visit pins for most queries.
    u = int(q[0])
    visits = orc.walk_visits(off, col, wl.num_pins, 77, u, walks, hops)[0]
    vals, cnts = np.unique(visits[(visits >= 0) & (visits != u)], return_counts=True)
    assert np.sort(cnts)[::-1][hi - 1] >= 2, "rank 5000 should still be a repeated pin"


@pytest.mark.parametrize("pins,boards,walks,hops,lo,hi,k,nq", [
    (2000, 500, 20000, 1, 100, 1900, 5, 300),   # every pin ranked (D <= rank_hi), > 256 queries
    (60, 10, 65536, 4, 0, 10, 7, 20),            # counts above 4096: second count digit
    (300, 40, 8192, 4, 20, 200, 3, 50),          # threshold inside a count class
])
def test_global_table_small_graphs(orc, pins, boards, walks, hops, lo, hi, k, nq):
    base = synth.WORKLOADS["tiny"]
    wl = base.scaled(pins, boards, f"hn-{pins}")
    off, col, _ = synth.make_graph(wl)
    q = _queries(wl, nq, pins + walks)
    print(f"[case] hard negatives, global table P={pins} B={boards} W={walks} H={hops} "
          f"[{lo},{hi}) k={k} n={nq}", flush=True)
    got, steps = _gpu(off, col, wl.num_pins, wl.num_boards, q, k, 5, walks, hops, lo, hi)
    np.testing.assert_array_equal(got, orc.hard_negatives(off, col, wl.num_pins, 5, walks, hops,
                                                          q, lo, hi, k))
    want = sum(orc.walk_visits(off, col, wl.num_pins, 5, u, walks, hops)[1] for u in q.tolist())
    assert steps == want


def test_global_table_int64_offsets(orc, tiny):
    wl, off, col = tiny
    q = _queries(wl, 64, 41)
    print("[case] hard negatives, global table, int64 offsets", flush=True)
    got, _ = _gpu(off, col, wl.num_pins, wl.num_boards, q, 4, 8, 9000, 3, 50, 700,
                  offsets64=True)
    np.testing.assert_array_equal(got, orc.hard_negatives(off, col, wl.num_pins, 8, 9000, 3, q,
                                                          50, 700, 4))


def _fmix32(x):
    # MurmurHash3's 32-bit finaliser, as the kernel partitions pins by it.
    x ^= x >> 16
    x = (x * 0x85EBCA6B) & 0xFFFFFFFF
    x ^= x >> 13
    x = (x * 0xC2B2AE35) & 0xFFFFFFFF
    x ^= x >> 16
    return x


def test_global_table_partition_split(orc):
    # One board joined to 30,000 pins that all fall in the first of the three
    # hash partitions of 4096 walks x 5 landings: about 15,000 distinct pins in
    # one partition, more than the 12,288 LDS slots, so the kernel splits it by
    # its second hash and counts each part again; its landings also overflow
    # the partition's workspace bucket. The ranking must still equal the
    # oracle's.
    walks, hops = 4096, 5
    parts = (walks * hops + 8191) // 8192
    chosen = [v for v in range(1, 400_000) if (_fmix32(v) * parts) >> 32 == 0][:30_000]
    P = chosen[-1] + 1
    edges = [(0, 0)] + [(v, 0) for v in chosen]
    off, col = synth.csr_from_edges(P, 1, edges)
    q = np.array([0, chosen[7], chosen[123]], np.int32)
    lo, hi, k = 100, 8000, 16
    print(f"[case] hard negatives, partition split P={P} pins={len(chosen)}", flush=True)
    got, steps = _gpu(off, col, P, 1, q, k, 21, walks, hops, lo, hi)
    np.testing.assert_array_equal(got, orc.hard_negatives(off, col, P, 21, walks, hops, q,
                                                          lo, hi, k))
    visits = orc.walk_visits(off, col, P, 21, 0, walks, hops)[0]
    assert len(np.unique(visits[(visits >= 0) & (visits != 0)])) > 12_288
    # Every landing falls in that partition, more than its 12,288-landing
    # workspace bucket holds: the rest takes the overflow list.
    assert np.count_nonzero((visits >= 0) & (visits != 0)) > 12_288
