"""Pins of the oracle's LRU simulator (Algorithm 1 of WiSP, Sec. 3.2).

- The paper's DiT-MoE fault counts (Appendix F.1), which need no weights.
- Mattson's stack-distance property of LRU: on a stream of single references, the misses at cap C
  are exactly the references whose reuse distance exceeds C (or that are first touches).
- Set-step invariants: every expert of the last m steps stays resident when their union fits.
- Budget equal to all experts: only compulsory misses from cold, none once pre-populated.
"""
import json
import os

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "dit_moe_faults.json")


def _dit_counts(cap, N, blocks, steps):
    faults = hits = 0
    for _ in range(blocks):
        sim = oracle.LRU(N, cap)
        for _ in range(steps):
            for e in range(N):              # one reference per expert, ascending id
                r = sim.step([e])
                faults += r["misses"]
                hits += r["hits"]
    return faults, hits


def test_dit_moe_fault_counts_from_paper():
    g = json.load(open(GOLDEN))
    N, B, S = g["n_experts"], g["n_blocks"], g["n_steps"]
    for cap in range(1, N):
        assert _dit_counts(cap, N, B, S) == (g["below_working_set"]["faults"], g["below_working_set"]["hits"])
    ws = g["at_working_set"]
    assert _dit_counts(ws["cap"], N, B, S) == (ws["faults"], ws["hits"])


def _stack_distance_misses(stream, C):
    """Misses by Mattson's stack algorithm: recency stack, distance = depth of the reference."""
    stack = []
    misses = []
    for e in stream:
        if e in stack:
            depth = stack.index(e) + 1
            stack.remove(e)
        else:
            depth = None
        stack.insert(0, e)
        misses.append(depth is None or depth > C)
    return misses


@pytest.mark.parametrize("seed", range(6))
def test_singleton_stream_matches_stack_distance(seed):
    rng = np.random.default_rng(seed)
    N = 24
    # locality: a drifting hot set plus uniform noise
    stream = []
    hot = list(rng.choice(N, 6, replace=False))
    for t in range(600):
        if rng.random() < 0.05:
            hot[rng.integers(6)] = int(rng.integers(N))
        stream.append(int(hot[rng.integers(6)]) if rng.random() < 0.8 else int(rng.integers(N)))
    prev = None
    for C in range(1, N + 1):
        sim = oracle.LRU(N, C)
        got = [sim.step([e])["misses"] == 1 for e in stream]
        assert got == _stack_distance_misses(stream, C)
        total = sum(got)
        if prev is not None:
            assert total <= prev            # LRU inclusion: misses never grow with the cap
        prev = total


def _random_set_trace(rng, N, steps, refs, rho=0.8):
    """Sets of `refs` distinct ids with step-to-step carry-over."""
    cur = list(rng.choice(N, refs, replace=False))
    trace = []
    for _ in range(steps):
        keep = [e for e in cur if rng.random() < rho]
        pool = [e for e in range(N) if e not in keep]
        cur = keep + list(rng.choice(pool, refs - len(keep), replace=False))
        trace.append(np.array(cur, np.int32))
    return trace


@pytest.mark.parametrize("N,C,refs", [(128, 32, 8), (16, 4, 3), (8, 2, 2), (256, 56, 8), (8, 8, 2)])
def test_set_steps_invariants(N, C, refs):
    rng = np.random.default_rng(N * 1000 + C)
    trace = _random_set_trace(rng, N, 300, refs)
    sim = oracle.LRU(N, C)
    seen = set()
    history = []
    for t, ids in enumerate(trace):
        resident_before = sim.resident()
        r = sim.step(ids)
        R = set(int(e) for e in ids)
        assert r["hits"] + r["misses"] == len(R)
        assert set(r["miss_ids"].tolist()) == R - resident_before      # faults are exactly the absent ids
        assert list(r["miss_ids"]) == sorted(r["miss_ids"])           # assigned in ascending id
        assert R <= sim.resident()                                      # all of R resident after the step
        assert len(sim.resident()) <= C
        slots = [sim.slot(e) for e in sim.resident()]
        assert len(set(slots)) == len(slots) and all(0 <= s < C for s in slots)
        # compulsory misses: a first touch always misses
        for e in R - seen:
            assert e in r["miss_ids"]
        seen |= R
        # LRU window property: experts of the latest m steps stay resident while their union fits
        history.append(R)
        U = set()
        for m in range(1, len(history) + 1):
            U |= history[-m]
            if len(U) > C:
                break
            assert U <= sim.resident()


def test_victims_are_least_recently_used_then_lowest_slot():
    sim = oracle.LRU(8, 3)
    sim.step([5])          # slot 0, tick 1
    sim.step([2, 7])       # slots 1, 2, tick 2
    sim.step([5])          # tick 3 on slot 0
    r = sim.step([1])      # victims by tick: slots 1 (e2) and 2 (e7) tie at 2 -> slot 1
    assert list(r["miss_ids"]) == [1] and list(r["miss_slots"]) == [1]
    assert sim.slot(2) == -1 and sim.slot(7) == 2
    r = sim.step([3, 4])   # U excludes nothing in R; ticks: slot0=3, slot1=4, slot2=2 -> slots 2 then 0
    assert list(r["miss_ids"]) == [3, 4] and list(r["miss_slots"]) == [2, 0]


def test_budget_equal_to_all_experts():
    rng = np.random.default_rng(7)
    N = 16
    trace = _random_set_trace(rng, N, 200, 4)
    cold = oracle.LRU(N, N)
    total_miss = sum(cold.step(ids)["misses"] for ids in trace)
    assert total_miss == len(set(np.concatenate(trace).tolist()))     # compulsory only
    warm = oracle.LRU(N, N)
    warm.step(np.arange(N))                                             # pre-populate every expert
    assert sum(warm.step(ids)["misses"] for ids in trace) == 0


def test_oversized_union_chunks():
    sim = oracle.LRU(8, 2)
    sim.step([4, 6])                   # 4 -> slot 0, 6 -> slot 1
    r = sim.step([0, 6, 3, 4, 7])      # residents first (4, 6), then misses ascending (0, 3, 7)
    assert r["chunks"] == 3 and r["hits"] == 2 and r["misses"] == 3
    # chunk 1 = {4, 6} (hits), chunk 2 = {0, 3} evicts both, chunk 3 = {7} evicts the LRU of {0,3}
    assert list(r["miss_ids"]) == [0, 3, 7]
    assert list(r["miss_slots"]) == [0, 1, 0]
    assert sim.resident() == {3, 7}
    # no expert is fetched twice within a layer-step
    assert len(set(r["miss_ids"].tolist())) == r["misses"]


def test_resize_keeps_most_recent():
    sim = oracle.LRU(16, 6)
    for ids in ([0, 1], [2, 3], [4, 5], [1, 3]):
        sim.step(ids)
    # ticks: e0 1, e2 2, e4 3, e5 3, e1 4, e3 4
    sim.resize(3)
    assert sim.resident() == {1, 3, 4}           # two at tick 4, then tick-3 tie -> lower slot (e4)
    assert [sim.slot(e) for e in (1, 3, 4)] == [0, 1, 2]      # renumbered in old slot order
    sim.resize(10)
    assert sim.resident() == {1, 3, 4} and sim.cap == 10
    r = sim.step([7, 8, 9])
    assert r["misses"] == 3 and set(r["miss_slots"].tolist()) == {3, 4, 5}   # empty slots first
    with pytest.raises(ValueError):
        sim.resize(0)
    with pytest.raises(ValueError):
        sim.resize(17)
