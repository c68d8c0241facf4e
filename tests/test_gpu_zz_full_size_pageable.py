"""GPU parity at full size with pageable masters: the DeepSeek-V3-shaped (180.4 GB) decode workload,
whose masters exceed the pinned memory a process may hold on the test machines, so every fault is
staged through the pinned bounce ring.  (The Mixtral-8x7B-shaped workload has its own module.)

These are the longest GPU tests; they are collected after all the others.
"""
import numpy as np
import pytest

from parity import run_case as _run_case
from paper_2606_21868_amd.workloads import WORKLOADS

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu


def test_deepseek_decode_full_size_sampled():
    """The DeepSeek-V3-shaped workload at full size (16 layers x 256 fp8 experts + shared, 180.4 GB
    of masters, C = 56 from the 40 GB budget), all 256 steps: all routing and
    paging decisions, outputs at sampled points, resident bit-identity (C = N, 180 GB of slots).
    Pageable masters (above the pinned-memory limit of the test machines), so the host pager only."""
    wl = WORKLOADS["deepseek-v3-16l-decode"]
    rng = np.random.default_rng(2)
    pts = sorted({(int(s), int(l)) for s, l in zip(rng.integers(0, wl.steps, 6), rng.integers(0, wl.L, 6))})
    pts += [(0, 0), (wl.steps - 1, wl.L - 1)]
    _run_case(wl, wl.cap, wl.steps, sample_points=pts, pageable=True)
