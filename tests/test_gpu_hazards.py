"""GPU hazard tests of the host pager's slot reuse (Sec. 3.2, the exactness invariant): with victim
poisoning on, every slot chosen as a victim is overwritten with NaN bytes on the side stream right
after its write-after-read wait and before its fill.  A fill that overtook the slot's last read, or
an FFN read that overtook the slot's fill, would then put NaN into the outputs.  Each case runs with
poisoning on and off from cold tables: the outputs must be bit-identical and match the oracle, over
the single-step fills, chunked unions larger than C, the token-batch fills, the staged fills of
pageable masters, and speculative prefetch."""
import numpy as np
import pytest

from parity import check_run, log
from paper_2606_21868_amd import wisp
from paper_2606_21868_amd.workloads import WORKLOADS, degraded_hints

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

CASES = {
    # name: (workload, shape, cap, steps, pageable)
    "decode-tight-cap": ("qwen3-30b-a3b-decode", dict(L=3), 10, 24, False),
    "chunked-unions": ("mixtral-8x7b-decode", dict(L=2, d=512, I=1024), 2, 24, False),
    "token-batch": ("qwen3-30b-a3b-prefill", dict(L=2, T=128), 32, 1, False),
    "staged-pageable": ("qwen3-30b-a3b-decode", dict(L=2), 16, 16, True),
}


@pytest.mark.parametrize("name", list(CASES))
def test_poisoned_victims_leave_outputs_exact(name):
    wl_name, shape, cap, steps, pageable = CASES[name]
    wl = WORKLOADS[wl_name].with_(**shape)
    log(f"[case] victim poisoning {name}: {wl.name} {shape} C={cap} steps={steps}")
    run = wisp.DecodeRun(wl, device=0, steps=steps, pageable=pageable)
    try:
        run.generate()
        assert run.set_cap(cap) == cap
        plain = run.decode(record=True)
        run.ctx.masters_ready()
        run.ctx.reset_stats()
        run.ctx.debug_poison_victims(True)
        poisoned = run.decode(record=True)
        run.ctx.debug_poison_victims(False)
        assert int(poisoned["misses"].sum()) > 0
        assert not np.isnan(poisoned["y"]).any(), "a poisoned slot reached the outputs"
        assert np.array_equal(poisoned["y"].view(np.uint32), plain["y"].view(np.uint32))
        pts = [(s, l) for s in range(0, steps, max(1, steps // 4)) for l in range(wl.L)]
        _, _, _, worst, _ = check_run(run, poisoned, steps, pts, tokens=None if wl.T <= 4 else np.arange(0, wl.T, 9),
                                      cap=cap)
        log(f"  {int(poisoned['misses'].sum())} poisoned fills: outputs bit-identical to the unpoisoned run, "
            f"worst error vs the oracle {worst:.2e}")
    finally:
        run.close()


def test_poisoned_victims_with_speculative_prefetch():
    wl = WORKLOADS["qwen3-30b-a3b-decode"].with_(L=3)
    cap, steps = 12, 16
    run = wisp.DecodeRun(wl, device=0, steps=steps)
    try:
        run.generate()
        assert run.set_cap(cap) == cap
        plain = run.decode(record=True)
        run.ctx.masters_ready()
        run.ctx.debug_poison_victims(True)
        run.ctx.set_prefetch(wisp.PREFETCH_HINTS)
        hints = degraded_hints(plain["idx"], wl.N, 0.5, seed=1)
        poisoned = run.decode(record=True, hints=hints)
        run.ctx.set_prefetch(wisp.PREFETCH_OFF)
        run.ctx.debug_poison_victims(False)
        assert run.ctx.prefetch_stats()["issued"] > 0
        assert np.array_equal(poisoned["y"].view(np.uint32), plain["y"].view(np.uint32))
        log(f"  prefetch with poisoned victims: {run.ctx.prefetch_stats()['issued']} prefetch copies, outputs "
            f"bit-identical")
    finally:
        run.close()
