"""Host check of the kernels' launch shapes: tests/c/grid_check.cpp includes
the same grid header as the kernels (paper_2102_02888_amd/csrc/onebit_grid.h)
and enumerates whole launches, including strided worker walks that no
workload here is large enough to reach on the GPU."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_every_tile_and_item_is_taken_once(tmp_path):
    exe = str(tmp_path / "grid_check")
    subprocess.run(["g++", "-std=c++17", "-O2", "-Wall", "-Wextra", "-Werror",
                    "-I" + os.path.join(ROOT, "paper_2102_02888_amd", "csrc"),
                    os.path.join(ROOT, "tests", "c", "grid_check.cpp"), "-o", exe],
                   check=True, timeout=300)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stdout[-2000:]
    assert "grid_check: ok" in r.stdout


def test_parity_cases_reach_every_partial_tile_shape():
    """The packed worker pass splits each tile between two waves (sub-blocks
    0-1 and 2-3), so a segment's last tile can end inside wave 0's first
    sub-block (<= 256 elements), inside its second (257-512, wave 1 idle) or
    in wave 1's half (> 512).  The GPU parity cases must hold all three."""
    import oracle
    from test_gpu_parity import CASES
    kinds = set()
    for numel, n in CASES:
        L = oracle.Layout(numel, n)
        for b, e in zip(L.seg_begin, L.seg_end):
            tail = (int(e) - int(b)) % 1024
            if tail:
                kinds.add(0 if tail <= 256 else 1 if tail <= 512 else 2)
    assert kinds == {0, 1, 2}
