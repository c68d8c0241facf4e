"""GPU parity of the degenerate shapes the paged decode path admits, and of its argument errors.

Each shape case runs the full parity check of a paged decode from a cold table (routing, Algorithm 1
decisions against the simulator, gates and outputs against the oracle, the device pager where it
applies, bit identity with the fully resident run) at the edge of what the method allows: top-1
routing in a single slot, every expert routed every step, the largest expert count at the smallest
budget the device pager accepts, group-limited routing with one expert per group, with every group
kept, and with the kept groups exactly filling the top-k, and a shared expert with a chunked batch.
"""
import numpy as np
import pytest

from parity import log, run_case
from paper_2606_21868_amd import wisp
from paper_2606_21868_amd.workloads import ROUTE_SIGMOID_GROUP, ROUTE_SOFTMAX_RENORM, ROUTE_TOPK_SOFTMAX, WORKLOADS

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

SMALL = WORKLOADS["qwen3-30b-a3b-decode"].with_(L=2, d=256, I=128)


def test_top1_in_one_slot():
    # k = 1, C = 1: the smallest budget a single-token step runs in; each step evicts the previous
    # expert unless the router repeats it, and the renormalised gate is exactly 1
    wl = SMALL.with_(N=8, k=1)
    out = run_case(wl, 1, 48, check_all_outputs=True)
    assert np.all(out["w"] == 1.0)
    assert np.all(out["hits"] + out["misses"] == 1)
    log(f"  top-1 hit rate {out['hits'].mean():.3f}")


@pytest.mark.parametrize("route", [ROUTE_SOFTMAX_RENORM, ROUTE_TOPK_SOFTMAX])
def test_every_expert_every_step(route):
    # k = N: the routed set is every expert; at C = N only the first step faults
    wl = SMALL.with_(N=8, k=8, route=route)
    out = run_case(wl, 8, 12, check_all_outputs=True)
    assert np.all(np.sort(out["idx"], axis=-1) == np.arange(8))
    assert np.all(out["misses"][0] == 8) and int(out["misses"][1:].sum()) == 0


def test_largest_expert_count_at_minimum_cap():
    # N = 256 (the most the router's one-thread-per-expert selection takes), C = k = 8
    wl = SMALL.with_(N=256, k=8)
    out = run_case(wl, 8, 32, check_all_outputs=True)
    assert np.all(out["misses"][0] == 8)


@pytest.mark.parametrize("N,n_groups,topk_groups,k", [
    (32, 32, 6, 4),      # one expert per group: a group's score is that expert's sigmoid alone
    (64, 8, 8, 8),       # every group kept: plain sigmoid top-k
    (64, 16, 2, 8),      # kept groups hold exactly k experts: every allowed expert is selected
])
def test_group_limited_routing_edges(N, n_groups, topk_groups, k):
    wl = SMALL.with_(N=N, k=k, route=ROUTE_SIGMOID_GROUP, n_groups=n_groups, topk_groups=topk_groups)
    out = run_case(wl, max(k, N // 4), 32, check_all_outputs=True)
    if topk_groups * (N // n_groups) == k:
        # the selection is a union of whole groups
        gs = N // n_groups
        groups = out["idx"] // gs
        for g in groups.reshape(-1, k):
            assert all(np.count_nonzero(g == q) == gs for q in np.unique(g))


def test_shared_expert_with_chunked_batch():
    # a shared expert beside a batch of four whose routed union exceeds C = 5 (chunked steps); the
    # shared expert is always resident and never counted as a fault
    wl = SMALL.with_(N=16, k=4, T=4, has_shared=True)
    out = run_case(wl, 5, 24, check_all_outputs=True)
    assert out["chunks"].max() > 1


def test_device_pager_at_its_minimum_budget():
    # T = 4 tokens at C = T * k exactly: the smallest budget the device pager accepts
    wl = SMALL.with_(N=32, k=4, T=4)
    run_case(wl, 16, 24, check_all_outputs=True)


def test_token_count_and_pointer_errors_leave_state_untouched():
    wl = SMALL.with_(N=16, k=4, T=2)
    run = wisp.DecodeRun(wl, device=0, steps=6)
    try:
        run.generate()
        assert run.set_cap(6) == 6
        ref = run.decode(record=True)
        run.ctx.masters_ready()
        run.ctx.reset_stats()
        idx = torch.zeros((wl.L, wl.T, wl.k), dtype=torch.int32, device="cuda")
        w = torch.zeros((wl.L, wl.T, wl.k), dtype=torch.float32, device="cuda")
        y = torch.zeros((wl.L, wl.T, wl.d), dtype=torch.float32, device="cuda")
        x = run.x_dev[0]
        for T in (0, -1, wl.T + 1):
            for call in (lambda: run.ctx.decode_step(x, T, idx, w, y, run.stream),
                         lambda: run.ctx.route_topk(0, x[0], T, idx[0], w[0], stream=run.stream),
                         lambda: run.ctx.page_in(0, np.zeros((1, wl.k), np.int32), T)):
                with pytest.raises(wisp.WispError) as ei:
                    call()
                assert ei.value.status == wisp.E_INVAL, (T, ei.value)
        for bad in ((None, idx, w, y), (x, None, w, y), (x, idx, None, y), (x, idx, w, None)):
            with pytest.raises(wisp.WispError) as ei:
                run.ctx.decode_step(bad[0], 1, bad[1], bad[2], bad[3], run.stream)
            assert ei.value.status == wisp.E_INVAL
        for layer in (-1, wl.L):
            with pytest.raises(wisp.WispError) as ei:
                run.ctx.route_topk(layer, x[0], 1, idx[0], w[0], stream=run.stream)
            assert ei.value.status == wisp.E_INVAL
        assert all(run.ctx.slot_of(l, e) == -1 for l in range(wl.L) for e in range(wl.N))
        again = run.decode(record=True)
        assert np.array_equal(again["idx"], ref["idx"])
        assert np.array_equal(again["hits"], ref["hits"]) and np.array_equal(again["misses"], ref["misses"])
        assert np.array_equal(again["y"].view(np.uint32), ref["y"].view(np.uint32))
    finally:
        run.close()


def test_link_probe_engines():
    # both fill engines move the expert blobs at a plausible link rate; the compute-unit engine needs
    # pinned masters and an engine outside the two is rejected
    wl = SMALL.with_(N=16, k=4, d=2048, I=768)
    run = wisp.DecodeRun(wl, device=0, steps=1)
    try:
        run.generate(inputs=False)
        ce = run.ctx.probe_h2d(8, 3)
        cu = run.ctx.probe_h2d(8, 3, engine=wisp.LINK_CUS)
        log(f"  link probe: copy engine {ce:.1f} GB/s, compute units {cu:.1f} GB/s")
        assert 5 < ce < 200 and 5 < cu < 200
        with pytest.raises(wisp.WispError) as ei:
            run.ctx.probe_h2d(8, 3, engine=2)
        assert ei.value.status == wisp.E_INVAL
    finally:
        run.close()
    run = wisp.DecodeRun(wl, device=0, steps=1, pageable=True)
    try:
        run.generate(inputs=False)
        with pytest.raises(wisp.WispError) as ei:
            run.ctx.probe_h2d(8, 3, engine=wisp.LINK_CUS)
        assert ei.value.status == wisp.E_INVAL
    finally:
        run.close()


def test_read_floor_probe():
    # a plain streaming read: positive times at a plausible HBM rate, longer for four times the bytes
    small = wisp.probe_hbm_read(27_566_080, 100)
    large = wisp.probe_hbm_read(4 * 27_566_080, 100)
    log(f"  read floor: 27.6 MB in {small:.2f} us, 110.3 MB in {large:.2f} us per launch")
    for nbytes, us in ((27_566_080, small), (4 * 27_566_080, large)):
        rate = nbytes / (us * 1e-6) / 1e9
        assert 500 < rate < 8000, (nbytes, us, rate)
    assert large > small


def test_matrix_core_probe():
    # the register-only bf16 MFMA stream runs near the chip's dense peak (2.5 PFLOP/s at 2.4 GHz)
    tf = wisp.probe_mfma(3)
    log(f"  matrix cores: {tf:.0f} TFLOP/s dense bf16")
    assert 500 < tf < 2800, tf
    with pytest.raises(wisp.WispError) as ei:
        wisp.probe_mfma(0)
    assert ei.value.status == wisp.E_INVAL
