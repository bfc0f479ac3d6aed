"""GPU: the random-read calibration kernel (bench support) follows the chains
it documents -- every lane's reads land where a host replay of the same
hash chain says, for 4-, 8- and 16-byte elements, and it validates its
arguments on the device path too."""

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
