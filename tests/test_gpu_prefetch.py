"""GPU tests of speculative expert prefetch (Sec. 4, predictor of App. E) through the C ABI.

A paged decode from a cold table with prefetch off is checked against the oracle (routing, pager,
outputs).  The same steps are then run again from a cold table with prefetch on:
- PREDICTOR: each step's per-layer requests must be a valid top-`depth` of the oracle predictor's
  exact scores, replayed on the GPU's routing trace;
- HINTS: the true routing of each step, given before it (a perfect predictor), and the same with
  half of each step's ids replaced by experts it does not use (a predictor of precision 0.5).
In both, the outputs must be bit-identical to the prefetch-off run (prefetch changes residency, never
the arithmetic), and the hits, misses, prefetch copies and useful prefetches must equal the oracle's
Algorithm 1 simulator replaying the same routing and the same prefetch requests.
"""
from fractions import Fraction

import numpy as np
import pytest

import oracle
from oracle.predictor import CoActivation
from parity import check_run, log
from paper_2606_21868_amd import wisp
from paper_2606_21868_amd.workloads import WORKLOADS, degraded_hints

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu


def _valid_top(ids, exact, depth):
    ids = [int(e) for e in ids]
    positive = sorted((e for e in range(len(exact)) if exact[e] > 0), key=lambda e: (-exact[e], e))
    assert len(ids) == min(depth, len(positive)), (ids, positive[:depth])
    assert len(set(ids)) == len(ids)
    for a, b in zip(ids[:-1], ids[1:]):
        assert exact[a] > exact[b] or (exact[a] == exact[b] and a < b) or abs(float(exact[a] - exact[b])) < 1e-12
    if ids:
        cut = exact[ids[-1]]
        assert {e for e in positive if exact[e] > cut and float(exact[e] - cut) >= 1e-12} <= set(ids)


def _replay(wl, cap, idx, requests):
    """Oracle replay: per layer an Algorithm 1 simulator; before layer l of step s, prefetch
    requests[s][l]; then the layer-step.  Returns hits, misses [S, L], copies issued, useful ones."""
    S = idx.shape[0]
    sims = [oracle.LRU(wl.N, cap) for _ in range(wl.L)]
    unused = [set() for _ in range(wl.L)]
    hits = np.zeros((S, wl.L), np.int64)
    misses = np.zeros((S, wl.L), np.int64)
    issued = useful = 0
    for s in range(S):
        for l in range(wl.L):
            req = requests[s][l]
            if len(req):
                fi, _ = sims[l].prefetch(req)
                issued += fi.size
                unused[l] |= set(fi.tolist())
            routed = set(idx[s, l].ravel().tolist())
            useful += sum(1 for e in routed & unused[l] if sims[l].slot(e) >= 0)
            unused[l] = set()
            r = sims[l].step(idx[s, l].ravel())
            hits[s, l], misses[s, l] = r["hits"], r["misses"]
    return hits, misses, issued, useful


@pytest.mark.parametrize("cap", [12, 32])
def test_prefetch_keeps_bits_and_matches_the_oracle_replay(cap):
    wl = WORKLOADS["qwen3-30b-a3b-decode"].with_(L=4)
    steps, depth, horizon, gamma = 24, wl.k, 2, 0.5
    log(f"[case] prefetch {wl.name} L={wl.L} C={cap} steps={steps} depth={depth} horizon={horizon}")
    run = wisp.DecodeRun(wl, device=0, steps=steps)
    try:
        run.generate()
        assert run.set_cap(cap) == cap
        off = run.decode(record=True)
        pts = [(0, 0), (steps // 2, 1), (steps - 1, wl.L - 1)]
        check_run(run, off, steps, pts, cap=cap)
        log(f"  prefetch off: {int(off['misses'].sum())} faults, checked against the oracle")

        # the online predictor
        run.ctx.masters_ready()            # cold tables again
        run.ctx.reset_stats()
        pred = wisp.Predictor(wl.L, wl.N, horizon, gamma)
        run.ctx.set_prefetch(wisp.PREFETCH_PREDICTOR, pred, depth)
        on = run.decode(record=True, prefetch_log=True)
        run.ctx.set_prefetch(wisp.PREFETCH_OFF)
        assert np.array_equal(on["idx"], off["idx"])
        assert np.array_equal(on["y"].view(np.uint32), off["y"].view(np.uint32)), "prefetch changed output bits"
        ora = CoActivation(wl.L, wl.N, horizon=horizon, gamma=Fraction(gamma))
        for s in range(steps):
            for l in range(wl.L):
                if l == 0:
                    assert on["requests"][s][l].size == 0
                else:
                    _valid_top(on["requests"][s][l].tolist(), ora.scores(l), depth)
                ora.observe(l, on["idx"][s, l].ravel())
            ora.end_pass()
        h, m, issued, useful = _replay(wl, cap, on["idx"], on["requests"])
        st = run.ctx.prefetch_stats()
        assert np.array_equal(on["hits"], h) and np.array_equal(on["misses"], m)
        assert (st["issued"], st["useful"]) == (issued, useful)
        log(f"  predictor: {int(m.sum())} faults + {issued} prefetch copies ({useful} used); bits unchanged")

        # perfect hints: the step's own routing
        run.ctx.masters_ready()
        run.ctx.reset_stats()
        run.ctx.set_prefetch(wisp.PREFETCH_HINTS)
        hints = off["idx"].reshape(steps, wl.L, -1)
        perfect = run.decode(record=True, hints=hints, prefetch_log=True)
        run.ctx.set_prefetch(wisp.PREFETCH_OFF)
        assert np.array_equal(perfect["y"].view(np.uint32), off["y"].view(np.uint32))
        h, m, issued, useful = _replay(wl, cap, perfect["idx"], perfect["requests"])
        st = run.ctx.prefetch_stats()
        assert np.array_equal(perfect["hits"], h) and np.array_equal(perfect["misses"], m)
        assert int(m.sum()) == 0 and (st["issued"], st["useful"]) == (issued, useful) and useful == issued
        log(f"  perfect hints: no demand fault, {issued} prefetch copies, all used; bits unchanged")

        # hints at precision 0.5: half of each step's routed set replaced by experts it does not use
        run.ctx.masters_ready()
        run.ctx.reset_stats()
        run.ctx.set_prefetch(wisp.PREFETCH_HINTS)
        hints = degraded_hints(off["idx"], wl.N, 0.5, seed=cap)
        half = run.decode(record=True, hints=hints, prefetch_log=True)
        run.ctx.set_prefetch(wisp.PREFETCH_OFF)
        assert np.array_equal(half["y"].view(np.uint32), off["y"].view(np.uint32))
        for s in range(steps):
            for l in range(wl.L):
                assert sorted(half["requests"][s][l].tolist()) == sorted(int(e) for e in hints[s, l] if e >= 0)
                assert len(set(hints[s, l].tolist()) & set(off["idx"][s, l].ravel().tolist())) == wl.k // 2
        h, m, issued, useful = _replay(wl, cap, half["idx"], half["requests"])
        st = run.ctx.prefetch_stats()
        assert np.array_equal(half["hits"], h) and np.array_equal(half["misses"], m)
        assert (st["issued"], st["useful"]) == (issued, useful) and useful < issued
        log(f"  hints at precision 0.5: {int(m.sum())} faults + {issued} prefetch copies ({useful} used); "
            f"bits unchanged")
    finally:
        run.close()


def test_prefetch_api_errors():
    wl = WORKLOADS["tiny-fp32"].with_(L=2)
    run = wisp.DecodeRun(wl, device=0, steps=4)
    try:
        run.generate()
        with pytest.raises(wisp.WispError) as ei:
            run.ctx.prefetch(0, [1])                     # no budget yet
        assert ei.value.status == wisp.E_STATE
        run.set_cap(4)
        with pytest.raises(wisp.WispError) as ei:
            run.ctx.prefetch(0, [wl.N])
        assert ei.value.status == wisp.E_INVAL
        with pytest.raises(wisp.WispError) as ei:
            run.ctx.set_prefetch_hints(np.zeros((wl.L, 2), np.int32))   # mode is not HINTS
        assert ei.value.status == wisp.E_STATE
        wrong = wisp.Predictor(wl.L + 1, wl.N, 1, 0.5)
        with pytest.raises(wisp.WispError) as ei:
            run.ctx.set_prefetch(wisp.PREFETCH_PREDICTOR, wrong, 2)
        assert ei.value.status == wisp.E_INVAL
        # an explicit prefetch, then a page-in and forward that route to it: no fault
        run.ctx.prefetch(1, [5, 6])
        assert {run.ctx.slot_of(1, 5) >= 0, run.ctx.slot_of(1, 6) >= 0} == {True}
        x = run.x_dev[0, 1]
        idx = torch.zeros((1, wl.k), dtype=torch.int32, device=run.dev)
        w = torch.zeros((1, wl.k), dtype=torch.float32, device=run.dev)
        y = torch.zeros((1, wl.d), dtype=torch.float32, device=run.dev)
        ids = np.zeros(wl.k, np.int32)
        run.ctx.route_topk(1, x, 1, idx, w, ids, run.stream)
        st = run.ctx.page_in(1, ids, 1)
        with pytest.raises(wisp.WispError) as ei:
            run.ctx.prefetch(1, [0])                     # between a page-in and its forward
        assert ei.value.status == wisp.E_STATE
        run.ctx.moe_forward(1, x, 1, w, y, run.stream)
        run.stream.synchronize()
        routed = set(ids.tolist())
        assert st["misses"] == len(routed - {5, 6})
        assert run.ctx.prefetch_stats() == dict(issued=2, useful=len(routed & {5, 6}))
        # the device pager refuses to start while prefetch is on
        run.ctx.set_prefetch(wisp.PREFETCH_HINTS)
        with pytest.raises(wisp.WispError) as ei:
            run.ctx.set_pager(wisp.PAGER_DEVICE)
        assert ei.value.status == wisp.E_STATE
        run.ctx.set_prefetch(wisp.PREFETCH_OFF)
    finally:
        run.close()
