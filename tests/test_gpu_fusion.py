"""GPU tests of the fused decode kernels: the down projection fused with the gate-weighted combine
(single-token steps, both pagers) and the device pager's router logits fused with its selection and
Algorithm 1.

The same decode steps run with the fused kernels and with the separate ones, from cold tables at the
same cap: routing, gates, paging decisions and outputs must be bit-identical (the fused kernels
compute every logit, row and sum with the same operations in the same order), the fused kernel must
be the one that ran, and the fused outputs are checked against the oracle.
"""
import numpy as np
import pytest

from parity import check_run, check_slots_hold_masters, log
from paper_2606_21868_amd import wisp
from paper_2606_21868_amd.workloads import WORKLOADS

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

QWEN = WORKLOADS["qwen3-30b-a3b-decode"]


def _decode(run, fused, pager=wisp.PAGER_HOST):
    run.ctx.set_pager(wisp.PAGER_HOST)
    run.ctx.masters_ready()                 # cold tables
    run.ctx.reset_stats()
    run.ctx.set_fusion(fused)
    run.ctx.set_pager(pager)
    run.ctx.reset_kernel_times()
    run.ctx.set_profiling((1 << wisp.K_DOWN_COMBINE) | (1 << wisp.K_FFN_DOWN) | (1 << wisp.K_COMBINE))
    out = run.decode(record=True)
    run.ctx.set_profiling(0)
    out["fused_launches"] = run.ctx.kernel_times(wisp.K_DOWN_COMBINE)["launches"]
    out["down_launches"] = run.ctx.kernel_times(wisp.K_FFN_DOWN)["launches"]
    out["combine_launches"] = run.ctx.kernel_times(wisp.K_COMBINE)["launches"]
    return out


@pytest.mark.parametrize("shape,cap,steps", [
    (dict(L=3), 32, 24),                                   # the benchmarked layer shape
    (dict(L=3), 12, 16),                                   # tight cap: most experts fault every step
    (dict(L=2, d=256, I=128, N=16, k=4), 6, 40),           # small widths, several tiles per row block
    (dict(L=2, d=384, I=128, N=24, k=6), 9, 40),           # 384 = 3 x 128: ragged against the 64-lane tile
])
def test_fused_matches_separate_kernels_and_oracle(shape, cap, steps):
    wl = QWEN.with_(**shape)
    log(f"[case] fusion {wl.name} {shape} C={cap} steps={steps}")
    run = wisp.DecodeRun(wl, device=0, steps=steps)
    try:
        run.generate()
        assert run.set_cap(cap) == cap
        sep = _decode(run, False)
        fus = _decode(run, True)
        assert sep["fused_launches"] == 0 and sep["combine_launches"] == steps * wl.L and sep["down_launches"] > 0
        assert fus["fused_launches"] == steps * wl.L and fus["down_launches"] == 0 and fus["combine_launches"] == 0
        if cap >= wl.k:
            dev = _decode(run, True, wisp.PAGER_DEVICE)
            assert dev["fused_launches"] == steps * wl.L and dev["combine_launches"] == 0
            assert np.array_equal(dev["idx"], sep["idx"]) and np.array_equal(dev["w"].view(np.uint32), sep["w"].view(np.uint32))
            assert np.array_equal(dev["hits"], sep["hits"]) and np.array_equal(dev["misses"], sep["misses"])
            assert np.array_equal(dev["y"].view(np.uint32), sep["y"].view(np.uint32)), "device pager: bits differ"
            assert check_slots_hold_masters(run) > 0   # the faults' blobs filled by the device-planned gate/up
            sep_dev = _decode(run, False, wisp.PAGER_DEVICE)
            assert sep_dev["fused_launches"] == 0
            assert np.array_equal(sep_dev["y"].view(np.uint32), sep["y"].view(np.uint32))
            assert check_slots_hold_masters(run) > 0
        assert np.array_equal(fus["idx"], sep["idx"])
        assert np.array_equal(fus["hits"], sep["hits"]) and np.array_equal(fus["misses"], sep["misses"])
        assert np.array_equal(fus["y"].view(np.uint32), sep["y"].view(np.uint32)), "fused down+combine changed bits"
        pts = [(s, l) for s in range(0, steps, max(1, steps // 6)) for l in range(wl.L)]
        _, _, _, worst, _ = check_run(run, fus, steps, pts, cap=cap)
        log(f"  fused == separate bit for bit over {steps * wl.L} layer-steps, both pagers; worst row-relative "
            f"error vs oracle {worst:.2e}")
    finally:
        run.close()


def test_fused_resident_and_repeated_launches():
    # all experts resident (every expert in the first gate/up launch), fused and separate alike; then
    # paging again at a small cap
    wl = QWEN.with_(L=2, d=256, I=128, N=16, k=4)
    steps = 64
    run = wisp.DecodeRun(wl, device=0, steps=steps)
    try:
        run.generate()
        assert run.set_cap(wl.N) == wl.N
        run.ctx.preload()
        run.ctx.set_fusion(True)
        res = run.decode(record=True)
        assert int(res["misses"].sum()) == 0
        run.ctx.set_fusion(False)
        sep = run.decode(record=True)
        assert np.array_equal(res["y"].view(np.uint32), sep["y"].view(np.uint32))
        assert run.set_cap(5) == 5
        run.ctx.masters_ready()
        run.ctx.set_fusion(True)
        paged = run.decode(record=True)
        assert np.array_equal(paged["y"].view(np.uint32), sep["y"].view(np.uint32))
    finally:
        run.close()
