"""GPU parity of the token-batch (prefill) path through the C ABI, against the oracle.

A prefill step routes a batch of prompt tokens per layer; the union of their experts exceeds the
cap, so each layer-step is several chunked Algorithm 1 steps, and the expert FFN runs as grouped
GEMMs on the matrix cores (the pairs ordered by expert on the device).  Checked as in decode:
routing and per-expert gates, hit/miss/chunk counts against the oracle's simulator, outputs within
the bf16 tolerance, and bit-identity with the fully resident run (C = N).
"""
import numpy as np
import pytest

from parity import log, run_case
from paper_2606_21868_amd import wisp
from paper_2606_21868_amd.workloads import WORKLOADS

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu


def test_prefill_qwen3_shape_reduced():
    # the prefill layer shape (d=2048, I=768, 128 experts top-8, C=32) at 2 layers x 128 tokens:
    # ~8 rows per expert, four chunks per layer-step
    wl = WORKLOADS["qwen3-30b-a3b-prefill"].with_(L=2, T=128)
    out = run_case(wl, 32, 1, check_all_outputs=True, expect_grouped=True)
    assert out["chunks"].min() >= 4


def test_prefill_multi_tile_ragged():
    # ~130 rows per expert (five 32-row slabs, the last ragged), K of two stages in the down GEMM (a
    # tile shorter than the prefetch distance), a ragged 16-token router tile (520 = 32 * 16 + 8), and
    # small caps (16 experts, C = 5 -> four chunks)
    wl = WORKLOADS["qwen3-30b-a3b-prefill"].with_(L=2, T=520, d=256, I=128, N=16, k=4)
    out = run_case(wl, 5, 1, check_all_outputs=True, expect_grouped=True)
    assert out["chunks"].min() >= 4


def test_prefill_experts_beyond_one_row_block():
    # ~260 rows per expert (8 experts, top-2 of 1040 tokens): an expert of more than 256 rows takes two
    # row blocks, each reading the expert's weights
    wl = WORKLOADS["qwen3-30b-a3b-prefill"].with_(L=2, T=1040, d=256, I=128, N=8, k=2)
    out = run_case(wl, 3, 1, check_all_outputs=True, expect_grouped=True)
    assert out["chunks"].min() >= 3


def test_prefill_pair_sort_in_two_launches():
    # 4200 tokens x top-8 of 256 experts = 33,600 pairs in 33 segments: 33 x 256 segment counts exceed
    # what the one-launch sort counts in LDS, so the counting launch runs first; ~131 rows per expert
    wl = WORKLOADS["qwen3-30b-a3b-prefill"].with_(L=1, T=4200, d=256, I=128, N=256, k=8)
    rng = np.random.default_rng(2)
    tokens = np.sort(np.concatenate([[0, wl.T - 1], rng.choice(np.arange(1, wl.T - 1), 126, replace=False)]))
    out = run_case(wl, 64, 1, sample_points=[(0, 0)], tokens=tokens, expect_grouped=True)
    assert out["chunks"].min() >= 4


def test_prefill_below_grouped_threshold():
    # a 12-token batch stays on the per-item GEMV path (one partial tile of the token-batch router)
    wl = WORKLOADS["qwen3-30b-a3b-prefill"].with_(L=2, T=12, d=256, I=128, N=16, k=4)
    run_case(wl, 5, 1, check_all_outputs=True, expect_grouped=False)


def test_prefill_router_rows_not_multiple_of_16():
    # 24 experts: the token-batch router takes its LDS-tiled FMA kernel instead of the matrix cores
    wl = WORKLOADS["qwen3-30b-a3b-prefill"].with_(L=2, T=40, d=256, I=128, N=24, k=4)
    run_case(wl, 7, 1, check_all_outputs=True, expect_grouped=True)


def test_prefill_full_size_sampled():
    """The prefill workload at full size (48 layers x 2048 tokens, 57.98 GB of masters, C = 32):
    every routing decision and paging count against the oracle; outputs of 24 sampled tokens at
    four layers; bit-identity with the fully resident run."""
    wl = WORKLOADS["qwen3-30b-a3b-prefill"]
    rng = np.random.default_rng(1)
    tokens = np.sort(np.concatenate([[0, wl.T - 1], rng.choice(np.arange(1, wl.T - 1), 22, replace=False)]))
    points = [(0, 0), (0, 17), (0, 30), (0, wl.L - 1)]
    out = run_case(wl, wl.cap, 1, sample_points=points, tokens=tokens, expect_grouped=True)
    assert int(out["misses"].sum()) == int((out["hits"] + out["misses"]).sum())   # a cold pass: all compulsory


def test_prefill_layer_calls_in_any_order():
    """wisp_route_topk orders a token batch's pairs by expert for the next forward of its layer.
    Routing both layers before paging either (on a second stream) leaves the first layer's order
    overwritten, so its forward orders the pairs itself: every order of the calls gives the bits of
    wisp_decode_step."""
    wl = WORKLOADS["qwen3-30b-a3b-prefill"].with_(L=2, T=64, d=256, I=128, N=16, k=4)
    log(f"[case] layer calls in any order {wl.name} L={wl.L} T={wl.T}")
    run = wisp.DecodeRun(wl, device=0, steps=1)
    try:
        run.generate()
        run.set_cap(wl.N)
        run.ctx.preload()
        ref = run.decode(record=True, steps=1)
        T, L, k = wl.T, wl.L, wl.k
        s2 = torch.cuda.Stream(device=run.dev)
        for order in ("route all, then page and forward", "route, page, forward per layer"):
            idx = torch.zeros((L, T, k), dtype=torch.int32, device=run.dev)
            w = torch.zeros((L, T, k), dtype=torch.float32, device=run.dev)
            y = torch.zeros((L, T, wl.d), dtype=torch.float32, device=run.dev)
            ids = [np.zeros(T * k, np.int32) for _ in range(L)]
            torch.cuda.synchronize(run.dev)
            if order.startswith("route all"):
                for l in range(L):
                    run.ctx.route_topk(l, run.x_dev[0, l], T, idx[l], w[l], ids[l], s2)
                run.stream.wait_stream(s2)
                for l in range(L):
                    run.ctx.page_in(l, ids[l], T)
                    run.ctx.moe_forward(l, run.x_dev[0, l], T, w[l], y[l], run.stream)
            else:
                for l in range(L):
                    run.ctx.route_topk(l, run.x_dev[0, l], T, idx[l], w[l], ids[l], run.stream)
                    run.ctx.page_in(l, ids[l], T)
                    run.ctx.moe_forward(l, run.x_dev[0, l], T, w[l], y[l], run.stream)
            run.stream.synchronize()
            assert np.array_equal(idx.cpu().numpy(), ref["idx"][0]), order
            assert np.array_equal(y.cpu().numpy().view(np.uint32), ref["y"][0].view(np.uint32)), order
            log(f"  {order}: bit-identical to wisp_decode_step")
    finally:
        run.close()


def test_prefill_counts_page_in_matches_ids_page_in():
    """wisp_decode_step pages a token batch in from the device's per-expert pair counts; the public
    route / page-in / forward sequence pages in from the routed ids.  From the same cold tables and
    with a budget below the union (chunked Algorithm 1 steps, faults in every layer), both make the
    same decisions (hits, misses, chunks per layer) and give the same output bits."""
    wl = WORKLOADS["qwen3-30b-a3b-prefill"].with_(L=2, T=64, d=256, I=128, N=16, k=4)
    log(f"[case] counts page-in against ids page-in {wl.name} L={wl.L} T={wl.T} N={wl.N} C=6")
    run = wisp.DecodeRun(wl, device=0, steps=1)
    try:
        run.generate()
        assert run.set_cap(6) == 6
        run.ctx.masters_ready()                       # cold tables
        ref = run.decode(record=True, steps=1)
        assert (ref["chunks"] > 1).all() and (ref["misses"] > 0).all()
        T, L, k = wl.T, wl.L, wl.k
        run.ctx.masters_ready()                       # cold tables again
        idx = torch.zeros((L, T, k), dtype=torch.int32, device=run.dev)
        w = torch.zeros((L, T, k), dtype=torch.float32, device=run.dev)
        y = torch.zeros((L, T, wl.d), dtype=torch.float32, device=run.dev)
        ids = [np.zeros(T * k, np.int32) for _ in range(L)]
        torch.cuda.synchronize(run.dev)
        for l in range(L):
            run.ctx.route_topk(l, run.x_dev[0, l], T, idx[l], w[l], ids[l], run.stream)
            st = run.ctx.page_in(l, ids[l], T)
            assert (st["hits"], st["misses"], st["chunks"]) == \
                (ref["hits"][0, l], ref["misses"][0, l], ref["chunks"][0, l]), l
            run.ctx.moe_forward(l, run.x_dev[0, l], T, w[l], y[l], run.stream)
        run.stream.synchronize()
        assert np.array_equal(idx.cpu().numpy(), ref["idx"][0])
        assert np.array_equal(y.cpu().numpy().view(np.uint32), ref["y"][0].view(np.uint32))
        log(f"  misses per layer {ref['misses'][0].tolist()}, chunks {ref['chunks'][0].tolist()}: same decisions and bits")
    finally:
        run.close()

