"""CPU tests of the parity rules the GPU tests apply (tests/parity.py), on routing traces built by
hand: exemptions are per token and only at near-ties, and every other mismatch fails."""
import types

import numpy as np
import pytest

import parity


def _wl(T=2, k=2, N=6):
    return types.SimpleNamespace(L=1, T=T, k=k, N=N)


def _trace(T=2, k=2, N=6):
    """One step, one layer: token scores with a clear top-k, the oracle's selection and margins."""
    scores = np.zeros((1, 1, T, N))
    scores[0, 0, :] = np.linspace(1.0, 0.5, N)        # expert 0 best, then 1, ...
    ora = np.tile(np.arange(k, dtype=np.int32), (1, 1, T, 1))
    margin = np.full((1, 1, T), scores[0, 0, 0, k - 1] - scores[0, 0, 0, k])
    gmargin = np.full((1, 1, T), np.inf)
    return scores, ora, margin, gmargin


def test_exact_match_passes():
    scores, ora, margin, gmargin = _trace()
    assert parity.check_routing(_wl(), ora.copy(), ora, margin, gmargin, scores) == (set(), set())


def test_near_tie_swap_exempts_only_that_token():
    scores, ora, margin, gmargin = _trace()
    scores[0, 0, 1, 2] = scores[0, 0, 1, 1] - 5e-7      # token 1: 2nd and 3rd within the tolerance
    margin[0, 0, 1] = 5e-7
    gpu = ora.copy()
    gpu[0, 0, 1, 1] = 2
    exempt, reordered = parity.check_routing(_wl(), gpu, ora, margin, gmargin, scores)
    assert exempt == {(0, 0, 1)} and reordered == set()


def test_mismatch_on_another_token_of_a_near_tie_step_fails():
    # token 1 has a near-tie, token 0 does not: a wrong choice on token 0 must not be hidden
    scores, ora, margin, gmargin = _trace()
    scores[0, 0, 1, 2] = scores[0, 0, 1, 1] - 5e-7
    margin[0, 0, 1] = 5e-7
    gpu = ora.copy()
    gpu[0, 0, 1, 1] = 2
    gpu[0, 0, 0, 1] = 3
    with pytest.raises(AssertionError):
        parity.check_routing(_wl(), gpu, ora, margin, gmargin, scores)


def test_near_tie_does_not_excuse_a_far_candidate():
    # the k-th/(k+1)-th are tied, but the GPU picked an expert far below them
    scores, ora, margin, gmargin = _trace()
    scores[0, 0, 0, 2] = scores[0, 0, 0, 1] - 5e-7
    margin[0, 0, 0] = 5e-7
    gpu = ora.copy()
    gpu[0, 0, 0, 1] = 5
    with pytest.raises(AssertionError):
        parity.check_routing(_wl(), gpu, ora, margin, gmargin, scores)


def test_rank_swap_of_near_equal_scores_is_a_valid_reorder():
    scores, ora, margin, gmargin = _trace()
    scores[0, 0, 0, 1] = scores[0, 0, 0, 0] - 1e-7
    gpu = ora.copy()
    gpu[0, 0, 0] = [1, 0]
    assert parity.check_routing(_wl(), gpu, ora, margin, gmargin, scores) == (set(), {(0, 0, 0)})
    # the same swap with clearly different scores is an error
    scores[0, 0, 0, 1] = scores[0, 0, 0, 0] - 1e-3
    with pytest.raises(AssertionError):
        parity.check_routing(_wl(), gpu, ora, margin, gmargin, scores)


def test_exempt_points_cover_every_exempt_token():
    ex = {(3, 1, 0), (3, 1, 2), (0, 4, 1)}
    assert parity.exempt_points(ex) == [(0, 4, [1]), (3, 1, [0, 2])]


def test_bound_is_per_token():
    wl = types.SimpleNamespace(L=48, T=2048, k=8, N=128)
    assert parity.routing_bound(1, wl) == 98
    assert parity.routing_bound(2, _wl()) == 2
