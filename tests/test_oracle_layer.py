"""Pins of the oracle's expert FFN and fully resident layer.

The reference here is the textbook form with library matrix products (numpy ``@``) over weights
decoded by PyTorch's own bf16 / float8_e4m3fn conversions, plus special cases whose answer is
known without computing the layer.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_21868_amd import datagen as dg
from paper_2606_21868_amd.workloads import WORKLOADS


def _decode_blob(blob, dtype, d, I):
    """(W1 [I,d], W3 [I,d], W2 [d,I]) as float64 via numpy / torch decoding."""
    n = d * I
    if dtype == dg.F32:
        w = blob.view(np.float32).astype(np.float64)
        return w[:n].reshape(I, d), w[n:2 * n].reshape(I, d), w[2 * n:].reshape(d, I)
    if dtype == dg.BF16:
        t = torch.from_numpy(blob.view(np.int16).copy()).view(torch.bfloat16).double().numpy()
        return t[:n].reshape(I, d), t[n:2 * n].reshape(I, d), t[2 * n:].reshape(d, I)
    codes = torch.from_numpy(blob[:3 * n].copy()).view(torch.float8_e4m3fn).double().numpy()
    sc = torch.from_numpy(blob[3 * n:].copy().view(np.int16)).view(torch.bfloat16).double().numpy()
    nb = (d // 128) * (I // 128)
    out = []
    for which, (rows, cols) in enumerate([(I, d), (I, d), (d, I)]):
        s = sc[which * nb:(which + 1) * nb].reshape(rows // 128, cols // 128)
        w = codes[which * n:(which + 1) * n].reshape(rows, cols)
        out.append(w * np.kron(s, np.ones((128, 128))))
    return tuple(out)


def _x_f64(x):
    if x.dtype == np.float32:
        return x.astype(np.float64)
    return torch.from_numpy(x.view(np.int16).copy()).view(torch.bfloat16).double().numpy()


def _textbook_expert(W1, W3, W2, x):
    a = W1 @ x
    b = W3 @ x
    return W2 @ (a / (1 + np.exp(-a)) * b)


@pytest.mark.parametrize("dtype,d,I", [(dg.F32, 256, 512), (dg.BF16, 256, 384), (dg.FP8, 256, 384)])
def test_expert_matches_textbook(dtype, d, I):
    blob = dg.expert_blob(0, 0, 3, dtype, d, I)
    W1, W3, W2 = _decode_blob(blob, dtype, d, I)
    xs = dg.decode_inputs(0, 1, 3, 1, d, dg.F32 if dtype == dg.F32 else dg.BF16)[0, :, 0]
    for x in xs:
        o, h = oracle.expert(blob, dtype, d, I, x, return_h=True)
        xv = _x_f64(x)
        want = _textbook_expert(W1, W3, W2, xv)
        np.testing.assert_allclose(o, want, rtol=1e-10, atol=1e-14)
        a = W1 @ xv
        np.testing.assert_allclose(h, a / (1 + np.exp(-a)) * (W3 @ xv), rtol=1e-10, atol=1e-16)


def test_silu_is_on_the_gate_branch():
    d, I = 256, 256
    blob = dg.expert_blob(0, 0, 0, dg.BF16, d, I)
    swapped = blob.copy()
    n2 = d * I * 2
    swapped[:n2], swapped[n2:2 * n2] = blob[n2:2 * n2], blob[:n2]
    x = dg.decode_inputs(0, 1, 1, 1, d, dg.BF16)[0, 0, 0]
    o = oracle.expert(blob, dg.BF16, d, I, x)
    o_sw = oracle.expert(swapped, dg.BF16, d, I, x)
    W1, W3, W2 = _decode_blob(blob, dg.BF16, d, I)
    xv = _x_f64(x)
    np.testing.assert_allclose(o, _textbook_expert(W1, W3, W2, xv), rtol=1e-10, atol=1e-14)
    assert np.abs(o - o_sw).max() > 1e-3 * np.abs(o).max()


def test_zero_down_projection_gives_zero():
    d, I = 256, 256
    blob = dg.expert_blob(0, 0, 0, dg.F32, d, I)
    blob.view(np.float32)[2 * d * I:] = 0
    x = dg.decode_inputs(0, 1, 1, 1, d, dg.F32)[0, 0, 0]
    assert np.all(oracle.expert(blob, dg.F32, d, I, x) == 0.0)


def _layer_inputs(wl, T, step_count, seed=0):
    blobs = [dg.expert_blob(seed, 0, e, wl.w_dtype, wl.d, wl.I) for e in range(wl.N)]
    Wr = dg.router_weights(seed, 0, wl.N, wl.d)
    xs = dg.decode_inputs(seed, 1, step_count, T, wl.d, wl.x_dtype)[0]
    shared = dg.expert_blob(seed, 0, dg.SHARED_EXPERT, wl.w_dtype, wl.d, wl.I) if wl.has_shared else None
    return blobs, Wr, xs, shared


def _textbook_layer(wl, blobs, Wr, x, shared):
    """Route with a library sort and combine with numpy products."""
    dec = [_decode_blob(b, wl.w_dtype, wl.d, wl.I) for b in blobs]
    xv = _x_f64(x)
    z = Wr.astype(np.float64) @ xv
    if wl.route == oracle.ROUTE_SOFTMAX_RENORM:
        p = np.exp(z - z.max()); p /= p.sum()
        order = np.lexsort((np.arange(wl.N), -p))[:wl.k]
        g = p[order] / p[order].sum()
    elif wl.route == oracle.ROUTE_TOPK_SOFTMAX:
        order = np.lexsort((np.arange(wl.N), -z))[:wl.k]
        e = np.exp(z[order] - z[order].max()); g = e / e.sum()
    else:
        s = 1 / (1 + np.exp(-z))
        gs = wl.N // wl.n_groups
        gam = np.array([np.sort(s[q * gs:(q + 1) * gs])[-2:].sum() for q in range(wl.n_groups)])
        keep = np.lexsort((np.arange(wl.n_groups), -gam))[:wl.topk_groups]
        allowed = np.concatenate([np.arange(q * gs, (q + 1) * gs) for q in keep])
        order = allowed[np.lexsort((allowed, -s[allowed]))[:wl.k]]
        g = s[order] / s[order].sum()
    y = sum(g[j] * _textbook_expert(*dec[order[j]], xv) for j in range(wl.k))
    if shared is not None:
        y = y + _textbook_expert(*_decode_blob(shared, wl.w_dtype, wl.d, wl.I), xv)
    return order, g, y


SMALL = {
    # the tiny workload at its full size
    "tiny-fp32": WORKLOADS["tiny-fp32"],
    # reduced widths of the other workloads, same routing and weight formats
    "qwen3-small": WORKLOADS["qwen3-30b-a3b-decode"].with_(L=1, d=256, I=128, N=16),
    "mixtral-small": WORKLOADS["mixtral-8x7b-decode"].with_(L=1, d=256, I=256),
    "deepseek-small": WORKLOADS["deepseek-v3-16l-decode"].with_(L=1, d=256, I=256, N=64),
}


@pytest.mark.parametrize("name", list(SMALL))
def test_layer_matches_textbook(name):
    wl = SMALL[name]
    T = wl.T
    blobs, Wr, xs, shared = _layer_inputs(wl, T, 4)
    for s in range(xs.shape[0]):
        x = xs[s]
        idx, g, y, margins, _ = oracle.moe_layer(wl.route, blobs, Wr, x, wl.k, wl.I, wl.w_dtype, shared,
                                                 wl.n_groups, wl.topk_groups)
        for t in range(T):
            order, gw, yw = _textbook_layer(wl, blobs, Wr, x[t], shared)
            assert list(idx[t]) == list(order)
            np.testing.assert_allclose(g[t], gw, rtol=1e-12)
            np.testing.assert_allclose(y[t], yw, rtol=1e-9, atol=1e-12 * np.abs(yw).max())
            assert margins[t] >= 0


def test_single_expert_layer_is_the_expert():
    wl = SMALL["qwen3-small"].with_(k=1)
    blobs, Wr, xs, _ = _layer_inputs(wl, 1, 1)
    idx, g, y, _, _ = oracle.moe_layer(wl.route, blobs, Wr, xs[0], 1, wl.I, wl.w_dtype)
    assert g[0, 0] == 1.0
    np.testing.assert_array_equal(y[0], oracle.expert(blobs[idx[0, 0]], wl.w_dtype, wl.d, wl.I, xs[0, 0]))


def test_shared_expert_adds_with_weight_one():
    wl = SMALL["deepseek-small"]
    blobs, Wr, xs, shared = _layer_inputs(wl, 1, 1)
    _, _, y_with, _, _ = oracle.moe_layer(wl.route, blobs, Wr, xs[0], wl.k, wl.I, wl.w_dtype, shared, 8, 4)
    _, _, y_wo, _, _ = oracle.moe_layer(wl.route, blobs, Wr, xs[0], wl.k, wl.I, wl.w_dtype, None, 8, 4)
    np.testing.assert_allclose(y_with[0] - y_wo[0], oracle.expert(shared, wl.w_dtype, wl.d, wl.I, xs[0, 0]),
                               rtol=1e-9, atol=1e-14)


def _textbook_gates_of_set(wl, Wr, xv, order):
    """Gates of a given routed set by the variant's rule, from numpy logits."""
    z = Wr.astype(np.float64) @ xv
    if wl.route == oracle.ROUTE_SOFTMAX_RENORM:
        p = np.exp(z - z.max())
        p /= p.sum()
        return p[order] / p[order].sum()
    if wl.route == oracle.ROUTE_TOPK_SOFTMAX:
        e = np.exp(z[order] - z[order].max())
        return e / e.sum()
    s = 1 / (1 + np.exp(-z))
    return s[order] / s[order].sum()


@pytest.mark.parametrize("name", list(SMALL))
def test_routed_layer_matches_textbook(name):
    """The layer evaluated on a routed set chosen by someone else (what a kernel may pick at a
    near-tie): the k-th expert swapped for the (k+1)-th candidate, and a random set in a random
    order.  Gates by the variant's rule over that set, combine in that order, from numpy."""
    wl = SMALL[name]
    blobs, Wr, xs, shared = _layer_inputs(wl, wl.T, 2)
    rng = np.random.default_rng(7)
    dec = [_decode_blob(b, wl.w_dtype, wl.d, wl.I) for b in blobs]
    dec_sh = _decode_blob(shared, wl.w_dtype, wl.d, wl.I) if shared is not None else None
    for s in range(xs.shape[0]):
        x = xs[s]
        own, g_own, y_own, _, _ = oracle.moe_layer(wl.route, blobs, Wr, x, wl.k, wl.I, wl.w_dtype, shared,
                                                   wl.n_groups, wl.topk_groups)
        # the oracle's own routing reproduces the plain layer
        g_r, y_r = oracle.moe_layer_routed(wl.route, blobs, Wr, x, own, wl.I, wl.w_dtype, shared)
        np.testing.assert_array_equal(g_r, g_own)
        np.testing.assert_array_equal(y_r, y_own)
        other = np.empty_like(own)
        for t in range(wl.T):
            sc = oracle.route(wl.route, Wr, x[t], wl.k, wl.n_groups, wl.topk_groups)[2]
            nxt = [e for e in np.lexsort((np.arange(wl.N), -sc)) if e not in own[t]][0]
            other[t] = own[t]
            other[t, -1] = nxt
            if s == 1:
                other[t] = rng.permutation(wl.N)[:wl.k]
        g, y = oracle.moe_layer_routed(wl.route, blobs, Wr, x, other, wl.I, wl.w_dtype, shared)
        for t in range(wl.T):
            xv = _x_f64(x[t])
            gw = _textbook_gates_of_set(wl, Wr, xv, other[t])
            np.testing.assert_allclose(g[t], gw, rtol=1e-12)
            assert abs(g[t].sum() - 1.0) < 1e-12
            yw = sum(gw[j] * _textbook_expert(*dec[other[t, j]], xv) for j in range(wl.k))
            if dec_sh is not None:
                yw = yw + _textbook_expert(*dec_sh, xv)
            np.testing.assert_allclose(y[t], yw, rtol=1e-9, atol=1e-12 * np.abs(yw).max())
            # a different set gives a different output: the given routing is really used
            assert np.abs(y[t] - y_own[t]).max() > 0


def test_routed_layer_rejects_bad_ids():
    wl = SMALL["qwen3-small"]
    blobs, Wr, xs, _ = _layer_inputs(wl, 1, 1)
    with pytest.raises(ValueError):
        oracle.moe_layer_routed(wl.route, blobs, Wr, xs[0], np.full((1, wl.k), wl.N), wl.I, wl.w_dtype)


@pytest.mark.parametrize("name", list(SMALL))
def test_route_gates_of_a_given_set(name):
    wl = SMALL[name]
    blobs, Wr, xs, shared = _layer_inputs(wl, wl.T, 1)
    rng = np.random.default_rng(3)
    for t in range(wl.T):
        idx, g, _, _, _ = oracle.route(wl.route, Wr, xs[0, t], wl.k, wl.n_groups, wl.topk_groups)
        np.testing.assert_array_equal(oracle.route_gates(wl.route, Wr, xs[0, t], idx), g)
        other = rng.permutation(wl.N)[:wl.k]
        np.testing.assert_allclose(oracle.route_gates(wl.route, Wr, xs[0, t], other),
                                   _textbook_gates_of_set(wl, Wr, _x_f64(xs[0, t]), other), rtol=1e-12)
