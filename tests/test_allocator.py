"""CPU tests of the expert <-> KV allocator (wisp_mvwsa.h): the library's miss curves, configurator
and dual-resize control law against the oracle (oracle/allocator.py), which is pinned here to the
mathematics (the LRU stack identity, closed-form optima) and to the paper's own numbers (Table 4)."""
import json
import math
import os

import numpy as np
import pytest

import oracle
from oracle import allocator as A
from paper_2606_21868_amd import wisp

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _ar_trace(rng, N, steps, k, keep=0.7):
    cur = list(rng.choice(N, k, replace=False))
    out = []
    for _ in range(steps):
        nxt = [e for e in cur if rng.random() < keep]
        pool = [e for e in range(N) if e not in nxt]
        nxt += list(rng.choice(pool, k - len(nxt), replace=False))
        cur = nxt
        out.append(np.array(cur, np.int32))
    return np.stack(out)


# ---------------------------------------------------------------- oracle pins
@pytest.mark.parametrize("seed", range(4))
def test_oracle_reuse_curve_is_lru_on_singleton_streams(seed):
    # one reference per step: the reuse-distance curve is exactly the LRU miss count at every cap
    # (the stack property of LRU), which the Algorithm 1 simulator computes step by step
    rng = np.random.default_rng(seed)
    N = 20
    stream = [int(v) for v in rng.integers(0, N, 400)]
    curve = A.reuse_curve([[e] for e in stream], N)
    assert curve[0] == len(stream)
    for C in range(1, N + 1):
        sim = oracle.LRU(N, C)
        assert curve[C] == sum(sim.step([e])["misses"] for e in stream), C


def test_oracle_reuse_curve_hand_example():
    # steps {0} {1} {0} {2} {1}: cold 0, 1, 2; 0 again after {1} (distance 1); 1 again after {0},{2} (2)
    assert A.reuse_curve([[0], [1], [0], [2], [1]], 3) == [5, 5, 4, 3]
    # set steps: duplicates count once and the experts of one step are one recency level
    # steps {0,2} {0}: 0 again with nothing between (distance 0, a hit at every cap >= 1)
    assert A.reuse_curve([[2, 0, 2], [0]], 3) == [3, 2, 2, 2]
    # steps {0,1} {2} {0}: distance 1; its previous step had one peer (1): upper bound counts 2
    assert A.reuse_curve([[0, 1], [2], [0]], 3) == [4, 4, 3, 3]
    assert A.reuse_curve_upper([[0, 1], [2], [0]], 3) == [4, 4, 4, 3]


def test_oracle_reuse_curve_brackets_algorithm1():
    # on set steps Algorithm 1's exact miss count lies between the two curves at every cap (the
    # peers of a step share its tick and are evicted among themselves by slot)
    rng = np.random.default_rng(3)
    for N, k in ((16, 4), (32, 8)):
        trace = _ar_trace(rng, N, 200, k)
        lo, hi = A.reuse_curve(trace, N), A.reuse_curve_upper(trace, N)
        for C in range(k, N + 1):
            sim = oracle.LRU(N, C)
            exact = sum(sim.step(s)["misses"] for s in trace)
            assert lo[C] <= exact <= hi[C], (N, k, C, lo[C], exact, hi[C])


def test_oracle_configure_closed_forms():
    N, a, b = 10, 100, 10
    B = 10 * a + 50 * b
    m_exp = [100 - 10 * C for C in range(N + 1)]      # every slot saves 10 misses
    flat_kv = [0.0] * 200
    # KV costs nothing: the optimum is every expert; the floor of 50 blocks then binds at C = 10,
    # and a floor of 60 blocks pulls it to C = 9
    r = A.configure(B, a, b, 50, 1.0, 1.0, m_exp, flat_kv)
    assert (r["cap"], r["kv_blocks"], r["floor_binding"]) == (10, 50, False)
    r = A.configure(B, a, b, 60, 1.0, 1.0, m_exp, flat_kv)
    assert (r["cap"], r["kv_blocks"], r["floor_binding"]) == (9, 60, True)
    # experts cost nothing: no expert slot
    r = A.configure(B, a, b, 0, 0.0, 1.0, m_exp, [float(200 - k) for k in range(200)])
    assert r["cap"] == 0
    # budget below the floor: infeasible
    assert A.configure(40 * b, a, b, 50, 1.0, 1.0, m_exp, flat_kv) is None


def test_oracle_configure_equimarginal():
    # convex curves: at the optimum one more byte is worth no more in either pool (Eq. 2, discretely)
    N, a, b = 64, 8, 1
    B = 64 * a + 256 * b
    m_exp = [1000.0 * math.exp(-C / 12.0) for C in range(N + 1)]
    m_kv = [800.0 * math.exp(-k / 90.0) for k in range(B // b + 1)]
    r = A.configure(B, a, b, 0, 1.0, 1.0, [int(round(v)) for v in m_exp], m_kv)
    C = r["cap"]
    T = lambda c: round(m_exp[c]) + m_kv[(B - c * a) // b]
    assert 0 < C < N
    assert T(C) <= T(C - 1) and T(C) <= T(C + 1)


def test_oracle_resize_law_table4():
    # the paper's live move (Sec. 5.3, Table 4; App. B): cap 32 -> 35, KV 2.79 -> 1.53 GiB
    g = json.load(open(os.path.join(GOLDEN, "dual_resize_table4.json")))
    a = g["layers"] * g["expert_bytes"]
    b = 1 << 20
    kv0 = int(round(g["kv_gib_before"] * (1 << 30))) // b
    B = g["cap_before"] * a + kv0 * b
    peak = int(g["peak_fraction"] * kv0)
    for h in (0.0, 0.1, 0.2):
        C, kv, move = A.resize_target(B, a, b, 0, h, 1, 128, 1, peak, g["cap_before"])
        assert C == g["cap_after"] and move
        assert abs(kv * b / (1 << 30) - g["kv_gib_after"]) <= g["kv_gib_after_tolerance"]
        assert C * a + kv * b <= B


def test_oracle_resize_law_rules():
    a, b = 100, 10
    B = 10 * a + 100 * b
    # the admission floor is kept even when the peak is small (Eq. 6)
    C, kv, _ = A.resize_target(B, a, b, 80, 0.0, 1, 20, 1, 5, 10)
    assert kv >= 80 and C == (B - 80 * b) // a
    # clip to C_max, and Eq. 8 gives the slack back to KV
    C, kv, _ = A.resize_target(B, a, b, 0, 0.0, 1, 12, 1, 0, 10)
    assert C == 12 and kv == (B - 12 * a) // b
    # dead zone: a one-expert move is suppressed with Delta = 2
    C, kv, move = A.resize_target(B, a, b, 0, 0.0, 1, 20, 2, 90, 10)
    assert C == 11 and not move
    assert A.resize_target(B, a, b, 0, 0.0, 1, 20, 1, 90, 10)[2]
    # C_min that does not fit
    assert A.resize_target(5 * a, a, b, 0, 0.0, 6, 20, 1, 0, 5) is None


# ---------------------------------------------------------------- library vs oracle
@pytest.mark.parametrize("N,k,steps", [(8, 2, 300), (128, 8, 256), (16, 4, 1), (32, 1, 500)])
def test_library_miss_curve_matches_oracle(N, k, steps):
    rng = np.random.default_rng(N + k)
    trace = _ar_trace(rng, N, steps, k)
    want = A.reuse_curve(trace, N)
    got = wisp.miss_curve(trace, N)
    assert got.tolist() == want
    lo, up = wisp.miss_curve(trace, N, upper=True)
    assert lo.tolist() == want and up.tolist() == A.reuse_curve_upper(trace, N)


def test_library_miss_curve_properties():
    rng = np.random.default_rng(5)
    N, k = 64, 8
    trace = _ar_trace(rng, N, 400, k)
    est = wisp.miss_curve(trace, N).astype(np.int64)
    assert est[0] == trace.size and est[N] == len(np.unique(trace))
    assert np.all(np.diff(est) <= 0)
    with pytest.raises(wisp.WispError):
        wisp.miss_curve(np.array([[0, N]], np.int32), N)


def test_library_configure_matches_oracle():
    rng = np.random.default_rng(11)
    for _ in range(200):
        N = int(rng.integers(1, 40))
        a = int(rng.integers(1, 50))
        b = int(rng.integers(1, 20))
        B = int(rng.integers(1, N * a + 400 * b))
        kv_min = int(rng.integers(0, 30))
        m_exp = np.sort(rng.integers(0, 1000, N + 1))[::-1].copy()
        m_kv = np.sort(rng.random(int(rng.integers(1, 80))) * 500)[::-1].copy()
        c_exp, c_kv = float(rng.random() * 3), float(rng.random() * 3)
        want = A.configure(B, a, b, kv_min, c_exp, c_kv, m_exp.tolist(), m_kv.tolist())
        if want is None:
            with pytest.raises(wisp.WispError):
                wisp.mvwsa_configure(B, a, b, kv_min, c_exp, c_kv, m_exp, m_kv)
            continue
        got = wisp.mvwsa_configure(B, a, b, kv_min, c_exp, c_kv, m_exp, m_kv)
        assert (got["cap"], got["kv_blocks"], got["floor_binding"]) == (want["cap"], want["kv_blocks"],
                                                                        want["floor_binding"])
        assert got["f"] == pytest.approx(want["f"], rel=1e-12)
        assert got["latency"] == pytest.approx(want["latency"], rel=1e-12)


def test_library_resize_target_matches_oracle():
    rng = np.random.default_rng(13)
    for _ in range(300):
        a = int(rng.integers(1, 100))
        b = int(rng.integers(1, 30))
        B = int(rng.integers(a, 64 * a + 500 * b))
        kv_min = int(rng.integers(0, 40))
        h = float(rng.random())
        cmin = int(rng.integers(1, 8))
        cmax = int(rng.integers(cmin, 80))
        dz = int(rng.integers(0, 4))
        peak = int(rng.integers(0, 600))
        now = int(rng.integers(cmin, cmax + 1))
        want = A.resize_target(B, a, b, kv_min, h, cmin, cmax, dz, peak, now)
        if want is None:
            with pytest.raises(wisp.WispError):
                wisp.resize_target(B, a, b, kv_min, h, cmin, cmax, dz, peak, now)
            continue
        assert wisp.resize_target(B, a, b, kv_min, h, cmin, cmax, dz, peak, now) == want


@pytest.mark.parametrize("seed,dz,every", [(0, 1, 4), (3, 2, 6), (5, 3, 8), (7, 0, 5)])
def test_library_controller_matches_oracle_replay(seed, dz, every):
    from paper_2606_21868_amd.workloads import kv_occupancy_trace
    N, a, b, kv0 = 128, 28 << 20, 4 << 20, 600
    B = 32 * a + kv0 * b
    occ = kv_occupancy_trace([(3 * every, "tool"), (2 * every, "long"), (3 * every, "tool")], kv0, seed=seed)
    want = A.controller_replay(B, a, b, 50, 0.2, 1, N, dz, 32, kv0, occ, every)
    ctl = wisp.Controller(B, a, b, 50, 0.2, 1, N, dz, 32, kv0)
    got = []
    for s0 in range(0, occ.size, every):
        for t in range(s0, s0 + every):
            ctl.observe(int(occ[t]))
        c, k, m, p = ctl.barrier()
        got.append((s0 + every - 1, p, c, k, m))
    assert got == want
    assert ctl.barrier() == (want[-1][2], want[-1][3], 0, -1)       # nothing observed: no move
    ctl.close()


def test_library_controller_rejects_bad_arguments():
    with pytest.raises(wisp.WispError):
        wisp.Controller(100, 10, 1, 0, 0.2, 1, 8, 1, 20, 0)            # split beyond the budget
    ctl = wisp.Controller(100, 10, 1, 0, 0.2, 1, 8, 1, 5, 50)
    with pytest.raises(wisp.WispError):
        ctl.observe(-1)
    ctl.close()


def test_kv_occupancy_trace_regimes():
    from paper_2606_21868_amd.workloads import kv_occupancy_trace
    occ = kv_occupancy_trace([(200, "tool"), (200, "long")], 1000, seed=1)
    assert occ.shape == (400,) and occ.dtype == np.int64
    assert occ[:200].max() < 0.7 * 1000 < occ[200:].min()
    assert np.array_equal(occ, kv_occupancy_trace([(200, "tool"), (200, "long")], 1000, seed=1))
