"""GPU: the calibration kernels (bench support) read what they document.

* Random reads: every lane's reads land where a host replay of the same hash
  chain says, for 4-, 8- and 16-byte elements.
* Random row gathers: the sum of every gathered word equals a host replay of
  the documented row positions, for 512-byte and 1 KB rows, with targets
  spanning several rounds of the grid.
"""

import ctypes

import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

M64 = (1 << 64) - 1


def _mix64(x):
    x ^= x >> 30
    x = (x * 0xbf58476d1ce4e5b9) & M64
    x ^= x >> 27
    x = (x * 0x94d049bb133111eb) & M64
    x ^= x >> 31
    return x


def _replay(words, eb, chains, steps, elements):
    per = eb // 4
    out = np.zeros(chains, np.uint32)
    for lane in range(chains):
        idx = _mix64((lane + 0x9e3779b97f4a7c15) & M64) & (elements - 1)
        acc = 0
        for s in range(steps):
            v = 0
            for k in range(per):
                v ^= int(words[idx * per + k])
            acc = (acc + v) & 0xFFFFFFFF
            idx = _mix64((v + s + lane) & M64) & (elements - 1)
        out[lane] = acc
    return out


@pytest.mark.parametrize("eb", [4, 8, 16])
def test_chains_match_host_replay(eb):
    from paper_1806_01973_amd import _lib
    L = _lib.lib()
    rng = np.random.default_rng(eb)
    nbytes = 4096 + 12  # the kernel uses the largest power of two of elements that fits
    words = rng.integers(0, 2**32, size=nbytes // 4, dtype=np.uint32)
    table = torch.from_numpy(words.view(np.int32)).cuda()
    chains, steps = 130, 9
    sink = torch.full((chains,), -1, dtype=torch.int32, device="cuda")
    print(f"[case] random-read calibration eb={eb}", flush=True)
    st = L.pinsage_profile_random_reads(table.data_ptr(), nbytes, eb, steps, sink.data_ptr(),
                                        chains, None)
    assert st == 0, L.pinsage_last_error()
    torch.cuda.synchronize()
    elements = 1
    while elements * 2 <= nbytes // eb:
        elements *= 2
    ref = _replay(words, eb, chains, steps, elements)
    np.testing.assert_array_equal(sink.cpu().numpy().view(np.uint32), ref)


def _mix64_np(x):
    x = x ^ (x >> np.uint64(30))
    x = x * np.uint64(0xbf58476d1ce4e5b9)
    x = x ^ (x >> np.uint64(27))
    x = x * np.uint64(0x94d049bb133111eb)
    return x ^ (x >> np.uint64(31))


@pytest.mark.parametrize("row_bytes,rows,targets,per", [(512, 1000, 3001, 50), (512, 777, 40000, 64),
                                                        (1024, 1000, 3001, 32), (1024, 513, 40000, 7)])
def test_gathers_match_host_replay(row_bytes, rows, targets, per):
    from paper_1806_01973_amd import _lib
    L = _lib.lib()
    rng = np.random.default_rng(row_bytes + per)
    wpr = row_bytes // 4
    words = rng.integers(0, 2**32, size=rows * wpr + 5, dtype=np.uint32)  # 20 bytes past the rows
    table = torch.from_numpy(words.view(np.int32)).cuda()
    sink = torch.zeros(1, dtype=torch.int32, device="cuda")
    seed = 0x1234_5678_9ABC
    print(f"[case] random-gather calibration {row_bytes} B rows, {rows} rows, {targets} x {per}",
          flush=True)
    st = L.pinsage_profile_random_gathers(table.data_ptr(), words.nbytes, row_bytes, targets, per,
                                          seed, sink.data_ptr(), None)
    assert st == 0, L.pinsage_last_error()
    torch.cuda.synchronize()
    with np.errstate(over="ignore"):
        keys = (np.uint64(seed) + np.uint64(64) * np.arange(targets, dtype=np.uint64)[:, None]
                + np.arange(per, dtype=np.uint64)[None, :])
        h = _mix64_np(keys) >> np.uint64(32)
        idx = (h * np.uint64(rows)) >> np.uint64(32)
    row_sums = words[:rows * wpr].reshape(rows, wpr).astype(np.uint64).sum(axis=1)
    ref = int(row_sums[idx.ravel()].sum()) & 0xFFFFFFFF
    assert int(sink.cpu().numpy().view(np.uint32)[0]) == ref
