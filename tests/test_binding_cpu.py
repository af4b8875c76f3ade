"""Host-side logic of the Python binding (no GPU): the per-chunk word ranges
that size a chunk owners' call, against brute force, and their per-call cost
on the 5,000-tensor stress layout; the paired gradient and error rows that
State allocates."""
import time

import numpy as np
import pytest
import torch

import oracle
import synth
from paper_2102_02888_amd.onebit import chunk_extent, chunk_word_ranges


def _brute_extent(L, sb, se):
    """Every owned non-empty segment visited one by one."""
    wlo, whi = -1, -1
    for k in range(L.K):
        for j in range(sb, se):
            q = k * L.n + j
            b, e = int(L.seg_begin[q]), int(L.seg_end[q])
            if e > b:
                wlo = b // 64 if wlo < 0 else min(wlo, b // 64)
                whi = max(whi, (e - 1) // 64)
    return wlo, whi, (L.K - 1) * L.n + se - 1


@pytest.mark.parametrize("numel,n", [
    ([1], 1), ([64], 3), ([5000, 70_001, 64, 0, 300], 4), ([0, 0, 10], 5),
    ([200, 1, 129, 64 * 33 + 1, 7], 33), ([10 ** 6], 32), ([0], 2),
])
def test_chunk_extent_matches_brute_force(numel, n):
    L = oracle.Layout(numel, n)
    lo, hi = chunk_word_ranges(L.seg_begin, L.seg_end, L.K, L.n)
    for sb in range(n):
        for se in range(sb + 1, n + 1):
            assert chunk_extent(lo, hi, L.K, L.n, sb, se) == _brute_extent(L, sb, se), (sb, se)


def test_chunk_extent_cost_on_stress_layout():
    """40,000 segments: the ranges are built once per plan and each chunk
    owners' call costs O(n) host work, far below one kernel's time."""
    wl = synth.get("stress")
    L = oracle.Layout(wl.numel, wl.n)
    t0 = time.perf_counter()
    lo, hi = chunk_word_ranges(L.seg_begin, L.seg_end, L.K, L.n)
    build_s = time.perf_counter() - t0
    assert build_s < 0.5, build_s
    calls = 2000
    t0 = time.perf_counter()
    for _ in range(calls):
        ext = chunk_extent(lo, hi, L.K, L.n, 0, L.n)
    per_call_ms = (time.perf_counter() - t0) * 1e3 / calls
    assert per_call_ms < 0.1, per_call_ms
    assert ext == _brute_extent(L, 0, L.n)
    for j in (0, 3, L.n - 1):
        assert chunk_extent(lo, hi, L.K, L.n, j, j + 1) == _brute_extent(L, j, j + 1)


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16, torch.float16])
def test_paired_rows_layout(dtype):
    """State's gradient and error rows share one allocation: row i holds D
    gradients and then D fp32 errors.  The views have the shapes and leading
    dimensions the ABI is given, every row starts 16-byte aligned, and a
    worker's two rows do not overlap each other or the next worker's."""
    from paper_2102_02888_amd.onebit import paired_rows
    n, D = 5, 192
    g, e = paired_rows(n, D, dtype, "cpu")
    gs = g.element_size()
    assert g.dtype == dtype and e.dtype == torch.float32
    assert g.shape == (n, D) and e.shape == (n, D)
    row_bytes = (gs + 4) * D
    assert g.stride() == (row_bytes // gs, 1) and e.stride() == (row_bytes // 4, 1)
    base = g.data_ptr()
    for i in range(n):
        g0, e0 = g[i].data_ptr() - base, e[i].data_ptr() - base
        assert g0 == i * row_bytes and e0 == i * row_bytes + gs * D
        assert g0 % 16 == 0 and e0 % 16 == 0
    g.fill_(1)
    assert float(e.abs().sum()) == 0.0
    e.fill_(2)
    assert bool((g == 1).all())
    with pytest.raises(ValueError):
        paired_rows(n, 100, dtype, "cpu")
    with pytest.raises(ValueError):
        paired_rows(n, 0, dtype, "cpu")
