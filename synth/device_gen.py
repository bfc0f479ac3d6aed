"""Seeded input generation on the GPU (torch) for graphs too large for numpy.

Same distributions as synth.graphs (pin degree Zipf(a) clipped to [1, hi],
board of each edge rank-Zipf(b) through a seeded rank -> id permutation,
distinct boards per pin, pin features N(0,1), board features = mean of their
pins, bf16 rounding for bf16 workloads), drawn with torch's generator on the
device, so the streams differ from the numpy generator's. Inputs only: no
arithmetic of the method is done here.
"""

from __future__ import annotations

import math
import warnings

import numpy as np
import torch


def _zeta(a: float, terms: int = 2_000_000) -> float:
    # Riemann zeta by direct summation plus the Euler-Maclaurin tail.
    k = np.arange(1, terms + 1, dtype=np.float64)
    n = float(terms)
    return float(np.sum(k ** -a) + n ** (1 - a) / (a - 1) - 0.5 * n ** -a)


def _draw_boards(gen, n, cdf, perm, B, device):
    u = torch.rand(n, generator=gen, dtype=torch.float64, device=device)
    rank = torch.searchsorted(cdf, u, right=True).clamp_(max=B - 1)
    return perm[rank]


def make_graph_device(wl, device="cuda", log=None):
    """Returns (offsets int64 [N+1], col int32 [nnz], num_edges) on `device`."""
    gen = torch.Generator(device=device)
    gen.manual_seed(1_000_003 * wl.seed + 11)
    P, B = wl.num_pins, wl.num_boards
    hi = min(wl.degree_hi, B)
    k = torch.arange(1, hi + 1, dtype=torch.float64, device=device)
    pmf = k ** (-wl.zipf_a) / _zeta(wl.zipf_a)
    cdf = torch.cumsum(pmf, 0)
    cdf[-1] = 1.0  # the mass above hi is clipped to hi
    u = torch.rand(P, generator=gen, dtype=torch.float64, device=device)
    deg = (torch.searchsorted(cdf, u, right=True) + 1).clamp_(max=hi)
    del u
    r = torch.arange(1, B + 1, dtype=torch.float64, device=device)
    bcdf = torch.cumsum(r ** (-wl.board_zipf), 0)
    bcdf /= bcdf[-1].clone()
    del r
    perm = torch.randperm(B, generator=gen, device=device)
    E = int(deg.sum().item())
    if log:
        log(f"{P} pins, {B} boards, {E} edges: drawing boards")
    pin = torch.repeat_interleave(torch.arange(P, dtype=torch.int64, device=device), deg)
    board = _draw_boards(gen, E, bcdf, perm, B, device)
    # Redraw duplicate (pin, board) pairs; each pass only revisits the edges of
    # pins that still hold a duplicate. After 64 passes drawn from the board
    # distribution, the duplicates left (a small part of the edges of the
    # heaviest pins, whose boards already hold most of the distribution's mass)
    # are redrawn uniformly over all boards.
    sel = torch.arange(E, dtype=torch.int64, device=device)
    for it in range(1000):
        key = pin[sel] * B + board[sel]
        ks, order = torch.sort(key, stable=True)
        dup = torch.zeros(len(sel), dtype=torch.bool, device=device)
        dup[1:] = ks[1:] == ks[:-1]
        del ks, key
        ndup = int(dup.sum().item())
        if ndup == 0:
            break
        if log and (it < 4 or it % 16 == 0):
            log(f"duplicate pass {it}: {ndup} redraws among {len(sel)} edges")
        idx = sel[order[dup]]
        del order, dup
        if it < 64:
            board[idx] = _draw_boards(gen, len(idx), bcdf, perm, B, device)
        else:
            board[idx] = torch.randint(0, B, (len(idx),), generator=gen, device=device)
        bad = torch.unique(pin[idx])
        sel = sel[torch.isin(pin[sel], bad)]
    else:  # pragma: no cover
        raise RuntimeError("duplicate redraw did not converge")
    del sel, bcdf, perm
    if log:
        log("building the CSR")
    # Pin rows: boards ascending within each pin.
    key, order = torch.sort(pin * B + board)
    del key
    pin_sorted_board = board[order]
    del order
    # Board rows: pins ascending within each board.
    key, order = torch.sort(board * P + pin)
    del key
    board_pins = pin[order]
    board_deg = torch.bincount(board, minlength=B)
    del order, pin, board
    offsets = torch.zeros(P + B + 1, dtype=torch.int64, device=device)
    offsets[1:P + 1] = torch.cumsum(deg, 0)
    offsets[P + 1:] = offsets[P] + torch.cumsum(board_deg, 0)
    col = torch.empty(2 * E, dtype=torch.int32, device=device)
    col[:E] = (pin_sorted_board + P).to(torch.int32)
    col[E:] = board_pins.to(torch.int32)
    return offsets, col, E


def make_features_device(wl, offsets, col, device="cuda", chunk_rows=1 << 22, log=None):
    """Node features [N, d_in] in the workload's storage dtype on `device`."""
    gen = torch.Generator(device=device)
    gen.manual_seed(1_000_003 * wl.seed + 22)
    P, B, d = wl.num_pins, wl.num_boards, wl.d_in
    dt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    x = torch.empty((P + B, d), dtype=dt, device=device)
    for r0 in range(0, P, chunk_rows):
        r1 = min(P, r0 + chunk_rows)
        x[r0:r1] = torch.randn((r1 - r0, d), generator=gen, dtype=torch.float32,
                               device=device).to(dt)
    if log:
        log("pin features drawn; averaging board features")
    # Board features: mean of the board's pins (fp32 sums over column slabs).
    b_off = (offsets[P:] - offsets[P]).to(torch.int64)
    b_col = col[int(offsets[P].item()):].to(torch.int64)
    cnt = torch.diff(b_off).to(torch.float32).clamp_(min=1.0)
    with warnings.catch_warnings():
        warnings.simplefilter("ignore")  # sparse CSR support is flagged as beta
        A = torch.sparse_csr_tensor(b_off, b_col, torch.ones(len(b_col), dtype=torch.float32,
                                                              device=device), size=(B, P))
    slab = int(max(1, min(d, (16 << 30) // (4 * max(P, 1)))))
    for c0 in range(0, d, slab):
        c1 = min(d, c0 + slab)
        sums = torch.sparse.mm(A, x[:P, c0:c1].float())
        x[P:, c0:c1] = (sums / cnt[:, None]).to(dt)
        del sums
        if log:
            log(f"board features: columns {c1}/{d}")
    return x
