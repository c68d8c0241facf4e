"""GPU test of wisp_route_topk_noalloc, the router entry point that allocates nothing (its scratch is
the library's fixed device array): called through the C ABI, its ids and gates must equal those of
wisp_route_topk (the context's own scratch, fusion on: the same kernels) bit for bit, on two calls in
a row, the second with a smaller input, for the one-launch path (T <= 4) and the two-launch path, in
every routing variant; sizes beyond the static scratch are rejected before any GPU call."""
import numpy as np
import pytest

from parity import log
from paper_2606_21868_amd import wisp
from paper_2606_21868_amd.workloads import WORKLOADS

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

SHAPES = {
    # (workload, reduced widths): only the router's N, d, k and variant matter here
    "softmax-renorm": ("qwen3-30b-a3b-decode", dict(L=1)),
    "topk-softmax": ("mixtral-8x7b-decode", dict(L=1, I=128, T=1)),
    "sigmoid-group": ("deepseek-v3-16l-decode", dict(L=1, I=256)),
}


def _route_both(run, x, T):
    wl = run.wl
    dev = run.dev
    ref_i = torch.full((T, wl.k), -1, dtype=torch.int32, device=dev)
    ref_w = torch.full((T, wl.k), -1.0, dtype=torch.float32, device=dev)
    got_i = torch.full((T, wl.k), -7, dtype=torch.int32, device=dev)
    got_w = torch.full((T, wl.k), -7.0, dtype=torch.float32, device=dev)
    s = run.stream
    with torch.cuda.stream(s):
        run.ctx.route_topk(0, x, T, ref_i, ref_w, stream=s)
        wisp.route_topk_noalloc(run.wr_dev[0], x, wl.x_dtype, T, wl.N, wl.d, wl.k, wl.route, wl.n_groups,
                                wl.topk_groups, got_i, got_w, stream=s)
    s.synchronize()
    return ref_i.cpu().numpy(), ref_w.cpu().numpy(), got_i.cpu().numpy(), got_w.cpu().numpy()


@pytest.mark.parametrize("variant", list(SHAPES))
@pytest.mark.parametrize("sizes", [(4, 1), (64, 9)])
def test_noalloc_router_matches_route_topk(variant, sizes):
    name, shape = SHAPES[variant]
    wl = WORKLOADS[name].with_(**shape)
    log(f"[case] route_topk_noalloc {variant} N={wl.N} d={wl.d} k={wl.k} T={sizes}")
    run = wisp.DecodeRun(wl, device=0, max_tokens=max(sizes), steps=1)
    try:
        run.generate(inputs=False)
        run.ctx.set_fusion(True)
        g = torch.Generator(device="cpu").manual_seed(11)
        for T in sizes:            # two calls in a row, the second with a smaller input
            xf = torch.randn((T, wl.d), generator=g, dtype=torch.float32)
            x = (xf if wl.x_dtype == wisp.F32 else xf.to(torch.bfloat16)).to(run.dev)
            ri, rw, gi, gw = _route_both(run, x, T)
            assert (ri >= 0).all() and (ri < wl.N).all()
            assert np.array_equal(gi, ri), f"T={T}: ids differ"
            assert np.array_equal(gw.view(np.uint32), rw.view(np.uint32)), f"T={T}: gates differ"
            log(f"  T={T}: ids and gates bit-identical to wisp_route_topk")
    finally:
        run.close()


def test_noalloc_router_rejects_beyond_its_scratch():
    dev = torch.device("cuda", 0)
    N, d = 256, 64
    wr = torch.zeros((N, d), dtype=torch.float32, device=dev)
    T = wisp.NOALLOC_MAX_LOGITS // N + 1
    x = torch.zeros((1, d), dtype=torch.float32, device=dev)
    idx = torch.zeros((1, 8), dtype=torch.int32, device=dev)
    w = torch.zeros((1, 8), dtype=torch.float32, device=dev)
    with pytest.raises(wisp.WispError) as ei:
        wisp.route_topk_noalloc(wr, x, wisp.F32, T, N, d, 8, 0, 1, 1, idx, w)
    assert ei.value.status == wisp.E_INVAL and "scratch" in str(ei.value)
    with pytest.raises(wisp.WispError) as ei:
        wisp.route_topk_noalloc(None, x, wisp.F32, 1, N, d, 8, 0, 1, 1, idx, w)
    assert ei.value.status == wisp.E_INVAL
