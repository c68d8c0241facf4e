"""Pins of the oracle's stored-value decoders and router against independent definitions.

Top-k selection is checked against a brute-force library sort; group-limited routing against an
enumeration of every group subset; gates against the identities the definitions imply.
"""
import itertools

import numpy as np
import pytest
import torch

import oracle


def test_bf16_decoder_all_codes():
    codes = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    ref = torch.from_numpy(codes.view(np.int16)).view(torch.bfloat16).double().numpy()
    got = np.array([oracle.bf16_value(c) for c in codes])
    r = ref
    both_nan = np.isnan(got) & np.isnan(r)
    assert np.array_equal(got[~both_nan], r[~both_nan])
    assert np.array_equal(np.isnan(got), np.isnan(r))


def test_e4m3_decoder_all_codes():
    codes = np.arange(256, dtype=np.uint8)
    ref = torch.from_numpy(codes).view(torch.float8_e4m3fn).double().numpy()
    got = np.array([oracle.e4m3_value(c) for c in codes])
    assert np.array_equal(np.isnan(got), np.isnan(ref))
    assert [c for c in codes if np.isnan(got[c])] == [0x7F, 0xFF]
    fin = ~np.isnan(ref)
    assert np.array_equal(got[fin], ref[fin])
    assert np.nanmax(got) == 448.0 and oracle.e4m3_value(0x01) == 2.0 ** -9


def _brute_topk(score, k, allowed=None):
    ids = np.arange(score.size)
    if allowed is not None:
        ids = ids[allowed]
    # library sort on (-score, id): score desc, id asc
    order = np.lexsort((ids, -score[ids]))
    return ids[order[:k]]


def _softmax(z):
    e = np.exp(z - z.max())
    return e / e.sum()


@pytest.mark.parametrize("seed", range(20))
@pytest.mark.parametrize("N,d,k", [(8, 16, 2), (16, 32, 4), (128, 64, 8)])
def test_softmax_renorm_matches_brute_force(seed, N, d, k):
    rng = np.random.default_rng(seed)
    Wr = rng.standard_normal((N, d)).astype(np.float32)
    x = rng.standard_normal(d).astype(np.float32)
    idx, g, sc, margin, _ = oracle.route(oracle.ROUTE_SOFTMAX_RENORM, Wr, x, k)
    z = Wr.astype(np.float64) @ x.astype(np.float64)
    p = _softmax(z)
    np.testing.assert_allclose(sc, p, rtol=1e-12)
    want = _brute_topk(p, k)
    assert list(idx) == list(want)
    np.testing.assert_allclose(g, p[want] / p[want].sum(), rtol=1e-12)
    assert abs(g.sum() - 1.0) < 1e-12 and (g > 0).all()
    assert np.all(np.diff(g) <= 0)  # rank order follows the score
    ps = np.sort(p)[::-1]
    assert abs(margin - (ps[k - 1] - ps[k])) < 1e-15


@pytest.mark.parametrize("seed", range(20))
def test_topk_softmax_matches_brute_force_and_equals_renorm(seed):
    rng = np.random.default_rng(100 + seed)
    N, d, k = 8, 64, 2
    Wr = rng.standard_normal((N, d)).astype(np.float32)
    x = rng.standard_normal(d).astype(np.float32)
    idx, g, sc, _, _ = oracle.route(oracle.ROUTE_TOPK_SOFTMAX, Wr, x, k)
    z = Wr.astype(np.float64) @ x.astype(np.float64)
    want = _brute_topk(z, k)
    assert list(idx) == list(want)
    np.testing.assert_allclose(g, _softmax(z[want]), rtol=1e-12)
    # softmax-then-renormalise over the chosen k equals softmax over the chosen logits
    idx0, g0, _, _, _ = oracle.route(oracle.ROUTE_SOFTMAX_RENORM, Wr, x, k)
    assert list(idx0) == list(idx)
    np.testing.assert_allclose(g0, g, rtol=1e-12)


def test_ties_break_to_lower_id():
    N, d, k = 8, 4, 3
    Wr = np.zeros((N, d), np.float32)
    Wr[[1, 4, 6], 0] = 1.0     # three equal top logits
    Wr[[2, 7], 0] = 0.5
    x = np.array([1, 0, 0, 0], np.float32)
    for v in (oracle.ROUTE_SOFTMAX_RENORM, oracle.ROUTE_TOPK_SOFTMAX):
        idx, g, _, margin, _ = oracle.route(v, Wr, x, k)
        assert list(idx) == [1, 4, 6]
        np.testing.assert_allclose(g, [1 / 3] * 3, rtol=1e-12)
    idx, _, _, margin, _ = oracle.route(oracle.ROUTE_TOPK_SOFTMAX, Wr, x, 2)
    assert list(idx) == [1, 4] and margin == 0.0


@pytest.mark.parametrize("seed", range(25))
def test_sigmoid_group_limited_brute_force(seed):
    rng = np.random.default_rng(200 + seed)
    N, d, k, G, KG = 256, 32, 8, 8, 4
    Wr = rng.standard_normal((N, d)).astype(np.float32)
    x = rng.standard_normal(d).astype(np.float32)
    idx, g, sc, margin, gmargin = oracle.route(oracle.ROUTE_SIGMOID_GROUP, Wr, x, k, G, KG)
    z = Wr.astype(np.float64) @ x.astype(np.float64)
    s = 1.0 / (1.0 + np.exp(-z))
    np.testing.assert_allclose(sc, s, rtol=1e-12)
    gs = N // G
    gamma = np.array([np.sort(s[q * gs:(q + 1) * gs])[-2:].sum() for q in range(G)])
    # enumerate all C(8,4) = 70 group subsets; with distinct group scores the kept subset is the
    # one with the largest total score
    best = max(itertools.combinations(range(G), KG), key=lambda S: sum(gamma[list(S)]))
    allowed = np.zeros(N, bool)
    for q in best:
        allowed[q * gs:(q + 1) * gs] = True
    want = _brute_topk(s, k, allowed)
    assert list(idx) == list(want)
    np.testing.assert_allclose(g, s[want] / s[want].sum(), rtol=1e-12)
    assert abs(g.sum() - 1) < 1e-12
    gsorted = np.sort(gamma)[::-1]
    assert abs(gmargin - (gsorted[KG - 1] - gsorted[KG])) < 1e-14
    # the selected experts all lie in kept groups, and at most k come from any group
    assert all(allowed[e] for e in idx)


def test_group_limit_changes_selection():
    # a case where the global top-8 of s is not admissible: group 0 holds one huge score only
    N, d, k, G, KG = 256, 8, 8, 8, 4
    Wr = np.zeros((N, d), np.float32)
    x = np.zeros(d, np.float32)
    x[0] = 1.0
    Wr[0, 0] = 10.0                      # expert 0 alone, group 0 second-best is 0.5
    for q in range(1, 5):                # groups 1..4 have two strong experts each
        Wr[q * 32, 0] = 2.0
        Wr[q * 32 + 1, 0] = 2.0
    idx, g, sc, _, _ = oracle.route(oracle.ROUTE_SIGMOID_GROUP, Wr, x, k, G, KG)
    s = 1 / (1 + np.exp(-10.0))
    s2 = 1 / (1 + np.exp(-2.0))
    # group 0 scores s(10) + 0.5 ~= 1.49999; groups 1..4 score 2*s(2) ~= 1.7616 -> group 0 dropped
    assert 0 not in idx
    assert sorted(idx) == [32, 33, 64, 65, 96, 97, 128, 129]
    assert 2 * s2 > s + 0.5
