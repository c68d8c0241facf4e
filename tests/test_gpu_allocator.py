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


def test_online_controller_follows_the_occupancy_trace():
    """The online controller (Sec. 3.5, App. B) over a KV-occupancy trace with regime shifts: at each
    drained barrier it takes the peak occupancy since the last one and applies the control law with
    its dead-zone.  The moves (in both directions, some suppressed by the dead-zone) equal the oracle's
    replay of the same trace; decode outputs across every move are bit-identical to the fully resident
    run and match the oracle; the budget holds after every barrier."""
    from oracle import allocator as A
    from parity import check_run
    from paper_2606_21868_amd import wisp
    from paper_2606_21868_amd.workloads import kv_occupancy_trace
    wl = WORKLOADS["qwen3-30b-a3b-decode"].with_(L=3)
    b, kv0, every, dz = 4 * MIB, 600, 6, 2
    occ = kv_occupancy_trace([(12, "tool"), (12, "long"), (12, "tool"), (12, "tool")], kv0, seed=3)
    steps = occ.size
    run = wisp.DecodeRun(wl, device=0, steps=steps)
    pool = ctl = None
    try:
        run.generate()
        a = wl.L * run.blob_bytes
        B = 32 * a + kv0 * b
        want = A.controller_replay(B, a, b, 50, 0.2, 1, wl.N, dz, 32, kv0, occ, every)
        # the trace moves both ways and the dead-zone suppresses a move somewhere
        caps = [32] + [r[2] for r in want]
        assert any(c1 > c0 for c0, c1 in zip(caps, caps[1:])) and any(c1 < c0 for c0, c1 in zip(caps, caps[1:]))
        suppressed = [r for r, c in zip(want, caps) if not r[4] and
                      A.resize_target(B, a, b, 50, 0.2, 1, wl.N, dz, r[1], c)[0] != c]
        assert suppressed
        run.set_cap(wl.N)
        run.ctx.preload()
        ref = run.decode(record=True)
        run.ctx.masters_ready()
        run.set_cap(32)
        pool = wisp.KvPool(b, kv0)
        ctl = wisp.Controller(B, a, b, 50, 0.2, 1, wl.N, dz, 32, kv0)
        outs, got = [], []
        for s0 in range(0, steps, every):
            outs.append(run.decode(record=True, steps=every, start=s0))
            for t in range(s0, s0 + every):
                ctl.observe(int(occ[t]))
            cap, kv, moved, peak = ctl.barrier(run.ctx, pool)
            assert run.ctx.cap() == cap and pool.blocks == kv and cap * a + kv * b <= B
            got.append((s0 + every - 1, peak, cap, kv, moved))
        assert got == want, (got, want)
        out = {k: np.concatenate([o[k] for o in outs]) for k in ("idx", "w", "y")}
        assert np.array_equal(out["y"].view(np.uint32), ref["y"].view(np.uint32)), "outputs changed across moves"
        pts = [(s, l) for s in range(0, steps, 5) for l in range(wl.L)]
        _, _, _, worst, _ = check_run(run, out, steps, pts)
        log(f"  caps {caps}: {sum(r[4] for r in want)} moves, {len(suppressed)} suppressed by the dead-zone; "
            f"moves equal the oracle replay; outputs bit-identical to resident, worst error {worst:.2e}")
    finally:
        if ctl is not None:
            ctl.close()
        if pool is not None:
            pool.close()
        run.close()


def test_miss_curves_of_the_gpu_trace_bracket_the_pager():
    """The expert miss curve (Sec. 3.2 reuse distances) computed by the library on the routing the GPU
    produced equals the oracle's curves on that trace, and per layer its lower and upper curves bracket
    the faults the pager actually took from cold at C = 8, 16, 32, 64 and 128."""
    from oracle import allocator as A
    from paper_2606_21868_amd import wisp
    wl = WORKLOADS["qwen3-30b-a3b-decode"].with_(L=2)
    steps = 96
    run = wisp.DecodeRun(wl, device=0, steps=steps)
    try:
        run.generate()
        curves = None
        trace = None
        for cap in (8, 16, 32, 64, 128):
            run.ctx.masters_ready()
            assert run.set_cap(cap) == cap
            out = run.decode(record=True)
            if trace is None:
                trace = out["idx"]
                curves = []
                for l in range(wl.L):
                    tl = trace[:, l].reshape(steps, -1)
                    lo, up = wisp.miss_curve(tl, wl.N, upper=True)
                    assert lo.tolist() == A.reuse_curve(tl.tolist(), wl.N)
                    assert up.tolist() == A.reuse_curve_upper(tl.tolist(), wl.N)
                    curves.append((lo, up))
            assert np.array_equal(out["idx"], trace)
            for l in range(wl.L):
                lo, up = curves[l]
                m = int(out["misses"][:, l].sum())
                assert int(lo[cap]) <= m <= int(up[cap]), (cap, l, int(lo[cap]), m, int(up[cap]))
            log(f"  C={cap:3d}: faults {out['misses'].sum(axis=0).tolist()} within the curves' bounds "
                f"{[(int(c[0][cap]), int(c[1][cap])) for c in curves]}")
    finally:
        run.close()
