"""GPU tests of wisp_set_budget: resizing the expert scratch at a drained barrier (WiSP Sec. 3.5,
App. B).  A shrink/grow cycle must keep outputs bit-identical to a fully resident run (the
paper's resize-cycle byte identity), follow the oracle simulator's resize rule (keep the most
recently used experts), keep every resident slot byte-equal to its master, and a failed grow must
leave the previous state untouched."""
import numpy as np
import pytest

import oracle
from parity import log
from paper_2606_21868_amd.workloads import WORKLOADS

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

WL = WORKLOADS["qwen3-30b-a3b-decode"].with_(L=3)
SCHEDULE = [(32, 10), (12, 10), (48, 10), (8, 10), (32, 8)]   # (cap, steps)


def _resident_reference(run, total):
    run.ctx.masters_ready()
    run.set_cap(WL.N)
    run.ctx.preload()
    return run.decode(record=True, steps=total, start=0)


def _check_slots_hold_masters(run, cap):
    for l in range(WL.L):
        for s in range(cap):
            e = run.ctx.expert_in_slot(l, s)
            if e >= 0:
                assert np.array_equal(run.ctx.read_slot(l, s, run.blob_bytes), run.master_blob(l, e)), (l, s, e)


@pytest.mark.parametrize("pager", ["host", "device"])
def test_resize_cycle_bit_identity_and_lru(pager):
    from paper_2606_21868_amd import wisp
    total = sum(n for _, n in SCHEDULE)
    log(f"[case] resize cycle {SCHEDULE} with the {pager} pager")
    run = wisp.DecodeRun(WL, device=0, steps=total)
    try:
        run.generate()
        ref = _resident_reference(run, total)
        run.ctx.set_pager(wisp.PAGER_HOST)
        run.ctx.masters_ready()
        sims = [oracle.LRU(WL.N, SCHEDULE[0][0]) for _ in range(WL.L)]
        start = 0
        free_before = None
        for i, (cap, n) in enumerate(SCHEDULE):
            free0 = torch.cuda.mem_get_info()[0]
            assert run.set_cap(cap) == cap
            free1 = torch.cuda.mem_get_info()[0]
            if i > 0 and cap < SCHEDULE[i - 1][0]:
                # a shrink returns the dropped slots' memory
                assert free1 - free0 >= (SCHEDULE[i - 1][0] - cap) * WL.L * run.blob_bytes * 0.9
            if i == 0:
                free_before = free1
                run.ctx.set_pager(wisp.PAGER_DEVICE if pager == "device" else wisp.PAGER_HOST)
            for sim in sims:
                if sim.cap != cap:
                    sim.resize(cap)
            # the tables after the resize: the most recently used experts, in slot order
            for l in range(WL.L):
                assert [run.ctx.slot_of(l, e) for e in range(WL.N)] == [sims[l].slot(e) for e in range(WL.N)]
            out = run.decode(record=True, steps=n, start=start)
            for s in range(n):
                for l in range(WL.L):
                    r = sims[l].step(out["idx"][s, l].ravel())
                    assert (out["hits"][s, l], out["misses"][s, l]) == (r["hits"], r["misses"]), (i, s, l)
            assert np.array_equal(out["idx"], ref["idx"][start:start + n])
            assert np.array_equal(out["y"].view(np.uint32), ref["y"][start:start + n].view(np.uint32)), \
                f"segment {i} (C={cap}) differs from the resident run"
            _check_slots_hold_masters(run, cap)
            log(f"  C={cap}: {n} steps bit-identical, LRU counts match, slots hold their masters")
            start += n
        assert free_before is not None
    finally:
        run.close()


def test_failed_grow_keeps_previous_state():
    from paper_2606_21868_amd import wisp
    run = wisp.DecodeRun(WL, device=0, steps=20)
    try:
        run.generate()
        ref = _resident_reference(run, 20)
        run.ctx.masters_ready()
        assert run.set_cap(16) == 16
        a = run.decode(record=True, steps=10, start=0)
        tables = [[run.ctx.slot_of(l, e) for e in range(WL.N)] for l in range(WL.L)]
        free0 = torch.cuda.mem_get_info()[0]
        for n in (1, 13, WL.L * 8):           # fail the first, a middle and the last of the 24 new slots
            run.ctx.debug_fail_slot_alloc(n)
            with pytest.raises(wisp.WispError) as ei:
                run.set_cap(24)
            assert ei.value.status == wisp.E_NOMEM
            assert run.ctx.cap() == 16
            assert [[run.ctx.slot_of(l, e) for e in range(WL.N)] for l in range(WL.L)] == tables
            assert torch.cuda.mem_get_info()[0] >= free0 - (64 << 20)   # nothing leaked
        for bad in (0, WL.blob * WL.L - 1, (WL.N + 1) * WL.L * WL.blob):
            with pytest.raises(wisp.WispError) as ei:
                run.ctx.set_budget(bad)
            assert ei.value.status == wisp.E_INVAL
            assert run.ctx.cap() == 16
        b = run.decode(record=True, steps=10, start=10)
        assert np.array_equal(a["y"].view(np.uint32), ref["y"][:10].view(np.uint32))
        assert np.array_equal(b["y"].view(np.uint32), ref["y"][10:].view(np.uint32))
        _check_slots_hold_masters(run, 16)
        # the device pager refuses a cap below one Algorithm 1 step per layer-step
        run.set_cap(8)
        run.ctx.set_pager(wisp.PAGER_DEVICE)
        with pytest.raises(wisp.WispError) as ei:
            run.set_cap(7)
        assert ei.value.status == wisp.E_INVAL and run.ctx.cap() == 8
    finally:
        run.close()


def test_api_order_errors():
    from paper_2606_21868_amd import wisp
    wl = WORKLOADS["tiny-fp32"]
    run = wisp.DecodeRun(wl, device=0, steps=2)
    try:
        run.generate()
        ids = np.zeros((1, wl.k), np.int32)
        with pytest.raises(wisp.WispError) as ei:          # no budget yet
            run.ctx.page_in(0, ids, 1)
        assert ei.value.status == wisp.E_STATE
        with pytest.raises(wisp.WispError) as ei:
            run.ctx.set_pager(wisp.PAGER_DEVICE)
        assert ei.value.status == wisp.E_STATE
        run.set_cap(wl.cap)
        with pytest.raises(wisp.WispError) as ei:          # forward without a page-in
            run.ctx.moe_forward(0, run.x_dev[0, 0], 1, run.x_dev[0, 0], run.x_dev[0, 0])
        assert ei.value.status == wisp.E_STATE
        with pytest.raises(wisp.WispError) as ei:          # id out of range: table untouched
            run.ctx.page_in(0, np.array([[0, wl.N]], np.int32), 1)
        assert ei.value.status == wisp.E_INVAL
        assert all(run.ctx.slot_of(0, e) == -1 for e in range(wl.N))
        st = run.ctx.page_in(0, np.array([[3, 5]], np.int32), 1)
        assert (st["hits"], st["misses"]) == (0, 2)
        with pytest.raises(wisp.WispError) as ei:          # a second page-in before the forward
            run.ctx.page_in(0, np.array([[3, 5]], np.int32), 1)
        assert ei.value.status == wisp.E_STATE
        with pytest.raises(wisp.WispError) as ei:          # resize with a pending page-in
            run.set_cap(wl.cap)
        assert ei.value.status == wisp.E_STATE
        w = torch.full((1, wl.k), 0.5, device="cuda")
        y = torch.zeros((1, wl.d), device="cuda")
        run.ctx.moe_forward(0, run.x_dev[0, 0], 1, w, y, run.stream)
        run.stream.synchronize()
        assert run.ctx.slot_of(0, 3) >= 0 and run.ctx.slot_of(0, 5) >= 0
    finally:
        run.close()
