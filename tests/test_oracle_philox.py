"""Pins for the oracle's counter-based generator (Philox4x32-10).

Two independent statements: the published known-answer vectors (Salmon et al.,
SC'11) and PyTorch's header-only Philox engine (a library routine, compiled
here with g++ and driven through its (seed, subsequence, offset) interface).
"""

import os
import subprocess

import numpy as np
import pytest

HERE = os.path.dirname(os.path.abspath(__file__))


def _kat_rows():
    rows = []
    with open(os.path.join(HERE, "golden", "philox4x32_10_kat.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            v = [int(t, 16) for t in line.split()]
            rows.append((v[0:4], v[4:6], v[6:10]))
    return rows


def test_philox_known_answers(orc):
    rows = _kat_rows()
    assert len(rows) == 3
    for ctr, key, want in rows:
        got = orc.philox4x32_10(ctr, key)
        assert [int(x) for x in got] == want


_TORCH_DRIVER = r"""
#include <ATen/core/PhiloxRNGEngine.h>
#include <cstdio>
#include <cstdint>
int main() {
  unsigned long long seed, sub, off;
  while (std::scanf("%llu %llu %llu", &seed, &sub, &off) == 3) {
    at::philox_engine e(seed, sub, off);
    unsigned a = e(), b = e(), c = e(), d = e();
    std::printf("%u %u %u %u\n", a, b, c, d);
  }
  return 0;
}
"""


def _torch_include():
    import torch
    return os.path.join(os.path.dirname(torch.__file__), "include")


def test_philox_matches_torch_engine(orc, tmp_path):
    inc = _torch_include()
    if not os.path.exists(os.path.join(inc, "ATen", "core", "PhiloxRNGEngine.h")):
        pytest.skip("torch Philox engine header not present")
    src = tmp_path / "drv.cpp"
    src.write_text(_TORCH_DRIVER)
    exe = tmp_path / "drv"
    subprocess.run(["g++", "-std=c++17", "-O1", "-I", inc, str(src), "-o", str(exe)], check=True)
    rng = np.random.default_rng(7)
    cases = rng.integers(0, 2**32, size=(300, 6), dtype=np.uint64)
    # torch's engine: key = (lo, hi) of seed; counter = (lo, hi) of offset, then
    # (lo, hi) of subsequence.
    lines = []
    for c in cases:
        seed = int(c[4]) | (int(c[5]) << 32)
        off = int(c[0]) | (int(c[1]) << 32)
        sub = int(c[2]) | (int(c[3]) << 32)
        lines.append(f"{seed} {sub} {off}")
    out = subprocess.run([str(exe)], input="\n".join(lines) + "\n", capture_output=True,
                         text=True, check=True).stdout.split("\n")
    for c, line in zip(cases, out):
        want = [int(t) for t in line.split()]
        got = orc.philox4x32_10([int(v) for v in c[:4]], [int(c[4]), int(c[5])])
        assert [int(x) for x in got] == want


def test_walk_word_stream_layout(orc):
    # Step s of walk w from node u reads word s % 4 of the block at counter
    # (u, w, s // 4, 0) under key (lo32(seed), hi32(seed)).
    seed = 0x0123456789ABCDEF
    key = [seed & 0xFFFFFFFF, seed >> 32]
    for (u, w, s) in [(0, 0, 0), (5, 3, 1), (17, 99, 6), (2**31 - 1, 7, 3)]:
        block = orc.philox4x32_10([u, w, s // 4, 0], key)
        assert orc.walk_word(seed, u, w, s) == int(block[s % 4])
