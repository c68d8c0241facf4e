"""GPU tests of the KV block pool and the drained-barrier move between the expert scratch and the KV
pool (App. B): the control law's target applied while decoding, outputs bit-identical across the
moves (property D2), the budget conserved, a failed grow rolled back."""
import numpy as np
import pytest

from parity import log
from paper_2606_21868_amd.workloads import WORKLOADS

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

MIB = 1 << 20


def test_kv_pool_tracks_its_size():
    from paper_2606_21868_amd import wisp
    torch.cuda.init()
    free0 = torch.cuda.mem_get_info()[0]
    pool = wisp.KvPool(MIB, 200)
    try:
        assert pool.blocks == 200
        used = free0 - torch.cuda.mem_get_info()[0]
        assert 200 * MIB <= used <= 200 * MIB + 64 * MIB, used
        pool.resize(70)              # frees the chunks left without a block: 128 blocks stay
        assert pool.blocks == 70
        used = free0 - torch.cuda.mem_get_info()[0]
        assert 70 * MIB <= used < 70 * MIB + 64 * MIB, used
        pool.resize(100)             # inside the slack: nothing allocated
        assert pool.blocks == 100 and free0 - torch.cuda.mem_get_info()[0] == used
        pool.resize(0)
        assert pool.blocks == 0
    finally:
        pool.close()
    assert torch.cuda.mem_get_info()[0] >= free0 - 8 * MIB


def test_dual_resize_cycle_keeps_bits_and_budget():
    from paper_2606_21868_amd import wisp
    wl = WORKLOADS["qwen3-30b-a3b-decode"].with_(L=3)
    b = 4 * MIB
    steps = 30
    run = wisp.DecodeRun(wl, device=0, steps=steps)
    pool = None
    try:
        run.generate()
        a = wl.L * run.blob_bytes
        kv0 = 600
        B = 32 * a + kv0 * b
        # fully resident reference
        run.set_cap(wl.N)
        run.ctx.preload()
        ref = run.decode(record=True)
        run.ctx.masters_ready()
        run.set_cap(32)
        pool = wisp.KvPool(b, kv0)
        outs = [run.decode(record=True, steps=10, start=0)]
        # a burst that used 40 % of the KV pool: the law moves the idle KV to experts (Eqs. 6-8)
        cap, kv, move = wisp.resize_target(B, a, b, 50, 0.2, 1, wl.N, 1, int(0.4 * kv0), 32)
        assert move and cap > 32 and cap * a + kv * b <= B
        wisp.dual_resize(run.ctx, pool, cap, kv)
        assert run.ctx.cap() == cap and pool.blocks == kv
        outs.append(run.decode(record=True, steps=10, start=10))
        # a long-context burst fills the pool: the law hands the bytes back to KV
        cap2, kv2, move2 = wisp.resize_target(B, a, b, 50, 0.2, 1, wl.N, 1, kv, cap)
        assert move2 and cap2 < cap and cap2 * a + kv2 * b <= B
        wisp.dual_resize(run.ctx, pool, cap2, kv2)
        assert run.ctx.cap() == cap2 and pool.blocks == kv2
        outs.append(run.decode(record=True, steps=10, start=20))
        y = np.concatenate([o["y"] for o in outs])
        assert np.array_equal(y.view(np.uint32), ref["y"].view(np.uint32)), "outputs changed across the moves"
        log(f"  C 32 -> {cap} -> {cap2}, KV {kv0} -> {kv} -> {kv2} blocks: outputs bit-identical, budget kept")
    finally:
        if pool is not None:
            pool.close()
        run.close()


def test_dual_resize_failed_grow_rolls_back():
    from paper_2606_21868_amd import wisp
    wl = WORKLOADS["qwen3-30b-a3b-decode"].with_(L=2)
    b = 4 * MIB
    run = wisp.DecodeRun(wl, device=0, steps=4)
    pool = None
    try:
        run.generate()
        run.set_cap(16)
        pool = wisp.KvPool(b, 300)
        run.decode(record=False)
        tables = [[run.ctx.slot_of(l, e) for e in range(wl.N)] for l in range(wl.L)]
        run.ctx.debug_fail_slot_alloc(3)           # the expert grow fails after the KV shrink
        with pytest.raises(wisp.WispError) as ei:
            wisp.dual_resize(run.ctx, pool, 20, 200)
        assert ei.value.status == wisp.E_NOMEM
        assert run.ctx.cap() == 16 and pool.blocks == 300
        assert [[run.ctx.slot_of(l, e) for e in range(wl.N)] for l in range(wl.L)] == tables
        with pytest.raises(wisp.WispError) as ei:
            wisp.dual_resize(run.ctx, pool, wl.N + 1, 10)
        assert ei.value.status == wisp.E_INVAL
    finally:
        if pool is not None:
            pool.close()
        run.close()
