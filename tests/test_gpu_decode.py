"""GPU parity of the paged decode path through the C ABI, against the oracle.

Each case generates the seeded weights straight into the library's pinned masters, runs
wisp_decode_step over every step from a cold slot table, and checks routing, paging and outputs
against the oracle; then it grows the budget to every expert (C = N), preloads, and checks that the
same kernels give bit-identical outputs with zero faults (the paper's byte-identity claim).
"""
import numpy as np
import pytest

import oracle
from parity import run_case as _run_case
from paper_2606_21868_amd.workloads import WORKLOADS

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu


def test_tiny_fp32_full():
    wl = WORKLOADS["tiny-fp32"]
    _run_case(wl, wl.cap, wl.steps, check_all_outputs=True)


def test_qwen3_shaped_layers_reduced_depth():
    # the benchmarked layer shape (d=2048, I=768, 128 experts, top-8, bf16, C=32), 3 layers x 24 steps
    wl = WORKLOADS["qwen3-30b-a3b-decode"].with_(L=3)
    _run_case(wl, 32, 24, check_all_outputs=True)


def test_ragged_bf16_shape():
    # widths that are not multiples of the 64-lane row tile: d=384 (48 chunks), I=192 (24 chunks)
    wl = WORKLOADS["qwen3-30b-a3b-decode"].with_(L=2, d=384, I=192, N=24, k=6)
    _run_case(wl, 7, 40, check_all_outputs=True)


def test_batch4_small_cap_chunks():
    # batched decode whose union exceeds C: chunked Algorithm 1 steps (reduced Mixtral widths)
    wl = WORKLOADS["mixtral-8x7b-decode"].with_(L=2, d=512, I=1024)
    out = _run_case(wl, 2, 24, check_all_outputs=True)
    assert out["chunks"].max() > 1


def test_qwen3_decode_full_size_sampled():
    """The benchmarked workload at full size and in the benchmarked launch configuration: every
    routing decision and every paging count against the oracle; outputs at 256 sampled (step, layer)
    points plus every exempt token."""
    wl = WORKLOADS["qwen3-30b-a3b-decode"]
    rng = np.random.default_rng(0)
    flat = rng.choice(wl.steps * wl.L, size=256, replace=False)
    pts = sorted({(int(f) // wl.L, int(f) % wl.L) for f in flat} | {(0, 0), (wl.steps - 1, wl.L - 1)})
    assert len(pts) >= 256
    _run_case(wl, wl.cap, wl.steps, sample_points=pts)


@pytest.mark.parametrize("T", [1, 4])
def test_mixtral_widths_pinned_one_layer(T):
    # the Mixtral widths (d=4096, I=14336: 28 16-byte loads per lane in the down rows) on one layer
    # with pinned masters; T = 1 runs the single-token kernels at these widths, T = 4 the chunked path
    wl = WORKLOADS["mixtral-8x7b-decode"].with_(L=1, T=T)
    _run_case(wl, 2, 6, check_all_outputs=True)


def test_qwen3_layers_pageable_masters():
    # the staged fill path (pageable masters through the pinned bounce ring): same decisions and bits
    wl = WORKLOADS["qwen3-30b-a3b-decode"].with_(L=2)
    _run_case(wl, 32, 16, check_all_outputs=True, pageable=True)


def test_deepseek_shaped_fp8_reduced():
    # fp8 E4M3 weights with 128x128 block scales, sigmoid group-limited routing, shared expert:
    # the DeepSeek-V3 layer shape (d=7168, I=2048, 256 experts, 8 groups) at 2 layers x 12 steps
    wl = WORKLOADS["deepseek-v3-16l-decode"].with_(L=2)
    _run_case(wl, 56, 12, check_all_outputs=True)


def test_fp8_conversion_all_codes():
    from paper_2606_21868_amd import wisp
    codes = torch.arange(256, dtype=torch.uint8, device="cuda")
    out = torch.empty(256, dtype=torch.float32, device="cuda")
    wisp.decode_fp8(codes, out, 256)
    torch.cuda.synchronize()
    got = out.cpu().numpy().astype(np.float64)
    want = np.array([oracle.e4m3_value(c) for c in range(256)])
    fin = ~np.isnan(want)
    assert np.array_equal(got[fin], want[fin])


def test_hbm_copy_kernel():
    from paper_2606_21868_amd import wisp
    src = torch.randint(0, 2**31 - 1, (1 << 20,), dtype=torch.int32, device="cuda")
    dst = torch.zeros_like(src)
    wisp.hbm_copy(src, dst, src.numel() * 4)
    torch.cuda.synchronize()
    assert torch.equal(src, dst)
