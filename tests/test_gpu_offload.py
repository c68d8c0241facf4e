"""GPU tests of the routing-blind static-offload arms (the comparison of the paper's iso-VRAM
evaluation, Sec. 5.2): at a VRAM expert budget they keep whole layers resident and stream every
other layer's experts in bulk each step (bulk) or read them over the link (zero-copy).  Each arm's
routing, gates and outputs are checked against the oracle on their own, and since it runs the same
router, expert and combine kernels as the pager, they must also equal the paged run's bit for bit."""
import numpy as np
import pytest

from parity import check_run, log
from paper_2606_21868_amd.workloads import WORKLOADS

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu


def _layer_bytes(run):
    stride = (run.blob_bytes + 4095) // 4096 * 4096
    return run.wl.N * stride


@pytest.mark.parametrize("mode,budget_layers,resident", [(0, 3, 1), (0, 2, 0), (0, 5, 5), (1, 3, 3), (1, 0, 0)])
def test_offload_matches_paged_bits(mode, budget_layers, resident):
    from paper_2606_21868_amd import wisp
    wl = WORKLOADS["qwen3-30b-a3b-decode"].with_(L=5, d=256, I=128, N=16, k=4)
    steps = 12
    log(f"[case] static offload ({'zero-copy' if mode else 'bulk'}), budget {budget_layers} layers, L={wl.L}")
    run = wisp.DecodeRun(wl, device=0, steps=steps)
    try:
        run.generate()
        assert run.set_cap(5) == 5
        paged = run.decode(record=True)
        r = run.ctx.offload_begin(budget_layers * _layer_bytes(run), mode)
        assert r == resident
        off = run.offload(record=True)
        _, exempt, _, worst, _ = check_run(run, off, steps, [(s, l) for s in range(steps) for l in range(wl.L)])
        log(f"  offload arm against the oracle: routing, gates, outputs at every layer-step (worst {worst:.2e})")
        assert np.array_equal(off["idx"], paged["idx"])
        assert np.array_equal(off["y"].view(np.uint32), paged["y"].view(np.uint32)), "offload arm changed bits"
        # a second run continues the copy sequence across calls
        off2 = run.offload(record=True, steps=4, start=2)
        assert np.array_equal(off2["y"].view(np.uint32), paged["y"][2:6].view(np.uint32))
        run.ctx.offload_end()
        log(f"  {resident} resident layers, {wl.L - resident} streamed: same routing and output bits as the pager")
    finally:
        run.close()


def test_offload_errors():
    from paper_2606_21868_amd import wisp
    wl = WORKLOADS["qwen3-30b-a3b-decode"].with_(L=3, d=256, I=128, N=16, k=4)
    run = wisp.DecodeRun(wl, device=0, steps=2)
    try:
        run.generate()
        lb = _layer_bytes(run)
        with pytest.raises(wisp.WispError) as ei:
            run.ctx.offload_step(run.x_dev[0], 1, run.x_dev[0], run.x_dev[0], run.x_dev[0])
        assert ei.value.status == wisp.E_STATE
        with pytest.raises(wisp.WispError) as ei:
            run.ctx.offload_begin(2 * lb - 1)
        assert ei.value.status == wisp.E_INVAL
        with pytest.raises(wisp.WispError) as ei:
            run.ctx.offload_begin(2 * lb, 7)
        assert ei.value.status == wisp.E_INVAL
        assert run.ctx.offload_begin(2 * lb) == 0
        with pytest.raises(wisp.WispError) as ei:
            run.ctx.offload_begin(2 * lb)
        assert ei.value.status == wisp.E_STATE
        run.ctx.offload_end()
        with pytest.raises(wisp.WispError) as ei:
            run.ctx.offload_end()
        assert ei.value.status == wisp.E_STATE
    finally:
        run.close()


def test_offload_full_size_bits():
    """The benchmarked shape at the C = 32 budget (12 layers of experts): bulk (10 resident layers, 2
    staging buffers, 38 streamed layers of 1.2 GB each) and zero-copy (12 resident layers): three
    steps each, bit-identical to the paged run."""
    from paper_2606_21868_amd import wisp
    wl = WORKLOADS["qwen3-30b-a3b-decode"]
    run = wisp.DecodeRun(wl, device=0, steps=3)
    try:
        run.generate()
        assert run.set_cap(wl.cap) == wl.cap
        paged = run.decode(record=True)
        for mode, resident in ((0, 10), (1, 12)):
            r = run.ctx.offload_begin(wl.cap * wl.L * run.blob_bytes, mode)
            assert r == resident
            off = run.offload(record=True)
            # streamed and resident layers both sampled: layers < r are resident, the rest streamed
            pts = [(0, 0), (0, r - 1), (1, r), (1, 30), (2, wl.L - 1), (2, 17)]
            _, _, _, worst, _ = check_run(run, off, 3, pts)
            assert np.array_equal(off["idx"], paged["idx"])
            assert np.array_equal(off["y"].view(np.uint32), paged["y"].view(np.uint32))
            run.ctx.offload_end()
            log(f"  full size, {'zero-copy' if mode else 'bulk'}: {r} resident layers; routing, gates and outputs at "
                f"{len(pts)} points against the oracle (worst {worst:.2e}); bit-identical to the paged run")
    finally:
        run.close()
