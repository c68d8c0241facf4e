"""ORACLE (test infrastructure, not part of the product): the expert <-> KV allocator of WiSP written
out plainly from the paper, for the tests of the library's allocator.

- reuse_curve: the expert miss curve m(C) from a routing trace by LRU reuse distances (Sec. 3.2,
  "Reuse-distance miss curves").  Algorithm 1 gives every expert of a step the same tick, so the
  reuse distance of a reference is counted at step level: the number of distinct experts referenced
  in the steps strictly between its previous reference and this one.  A reference misses at cap C iff
  it is a first reference or that distance is >= C.  Experts referenced after e are never evicted
  before e, so a distance >= C forces a miss under Algorithm 1, and a distance plus the other experts
  of e's previous step below C forces a hit: the curve is a lower bound on Algorithm 1's misses and
  reuse_curve_upper an upper bound, both exact on single-reference steps.
- configure: the startup configurator (Sec. 3.3-3.4): the split minimising the latency model
  T = c_exp m_exp(C) + c_kv m_kv(kappa) of Eq. 3, kappa = floor((B - C a) / b), then the two engine
  knobs of Eq. 5, whose cap respects the admission floor of Eq. 4.
- resize_target: the dual-resize control law of App. B (Eqs. 6-8) with the cap dead-zone.
"""
from __future__ import annotations

import math


def reuse_distances(trace, n_experts):
    """For every reference (each step's distinct ids): (D, peers) with D the number of distinct experts
    referenced in the steps strictly between its previous reference and this one (None for a first
    reference) and peers the number of other experts of that previous step."""
    last = [-1] * n_experts            # step of the latest reference
    size_at = []                       # distinct experts of each step
    out = []
    for t, step in enumerate(trace):
        ids = sorted(set(int(v) for v in step))
        for e in ids:
            p = last[e]
            if p < 0:
                out.append((None, 0))
            else:
                D = sum(1 for x in range(n_experts) if p < last[x] < t)
                out.append((D, size_at[p] - 1))
        for e in ids:
            last[e] = t
        size_at.append(len(ids))
    return out


def reuse_curve(trace, n_experts):
    """trace: iterable of per-step id collections.  Returns misses[C] for C = 0 .. n_experts: first
    references, plus references whose step-level reuse distance D is >= C."""
    ds = reuse_distances(trace, n_experts)
    return [sum(1 for D, _ in ds if D is None or D >= C) for C in range(n_experts + 1)]


def reuse_curve_upper(trace, n_experts):
    """misses[C] counting a reference also when D + (other experts of its previous step) >= C: an
    upper bound on Algorithm 1's misses (the peers of a step share its tick)."""
    ds = reuse_distances(trace, n_experts)
    return [sum(1 for D, q in ds if D is None or D + q >= C) for C in range(n_experts + 1)]


def configure(B, a, b, kv_min, c_exp, c_kv, m_exp, m_kv):
    """Eqs. 3-5.  m_exp[C] for C = 0..N; m_kv[kappa] for kappa = 0..len-1 (the last value beyond).
    The split f is the minimiser of the latency model of Eq. 3 over the caps the budget allows
    (kappa = floor((B - C a) / b)); Eq. 5 then clamps the cap by the admission floor of Eq. 4.  Ties
    in the latency go to the smaller cap.  Returns dict(cap, kv_blocks, kv_bytes, f, latency,
    floor_binding), or None when even C = 0 leaves less KV than the floor."""
    N = len(m_exp) - 1

    def latency(C):
        kappa = (B - C * a) // b
        return c_exp * m_exp[C] + c_kv * m_kv[min(kappa, len(m_kv) - 1)]

    best_T, best_C = None, None
    for C in range(0, min(N, B // a) + 1):
        T = latency(C)
        if best_T is None or T < best_T:
            best_T, best_C = T, C
    f = best_C * a / B
    # Eq. 5: C = min(floor(f B / a), floor((B - kappa_min b) / a)); floor(f B / a) is best_C itself
    if B < kv_min * b:
        return None
    C = min(best_C, (B - kv_min * b) // a)
    kappa = (B - C * a) // b
    return dict(cap=C, kv_blocks=kappa, kv_bytes=kappa * b, f=f, latency=latency(C), floor_binding=C < best_C)


def resize_target(B, a, b, kv_min, headroom, cap_min, cap_max, dead_zone, peak_blocks, cap_now):
    """App. B, Eqs. 6-8: kappa~ = max(kappa_min, ceil((1 + h) p)); C~ = clip(floor((B - kappa~ b) / a),
    C_min, C_max); kappa~ <- floor((B - C~ a) / b).  A move smaller than the dead-zone is suppressed.
    Returns (cap, kv_blocks, move), or None when C_min does not fit the budget."""
    kappa = max(kv_min, math.ceil((1.0 + headroom) * peak_blocks))
    C = (B - kappa * b) // a if B >= kappa * b else 0
    C = max(cap_min, min(cap_max, C))
    if C * a > B:                        # even C_min does not fit the budget
        return None
    kappa = (B - C * a) // b
    move = abs(C - cap_now) >= dead_zone and C != cap_now
    return C, kappa, move


def controller_replay(B, a, b, kv_min, headroom, cap_min, cap_max, dead_zone, cap0, kv0, occupancy, barrier_every):
    """The online controller of Sec. 3.5 / App. B replayed on a KV-occupancy trace: after each decode
    step t the blocks in use occupancy[t] are seen; after every barrier_every steps there is a drained
    barrier, where p is the largest occupancy since the previous barrier and the law's target (with its
    dead-zone) against the current split is applied when a move is due.  Returns one record per
    barrier: (step, p, cap, kv_blocks, moved) with the split in place after the barrier."""
    cap, kv = cap0, kv0
    out = []
    peak = None
    for t, occ in enumerate(occupancy):
        peak = occ if peak is None else max(peak, occ)
        if (t + 1) % barrier_every == 0:
            moved = 0
            r = resize_target(B, a, b, kv_min, headroom, cap_min, cap_max, dead_zone, peak, cap)
            if r is not None and r[2]:
                cap, kv, moved = r[0], r[1], 1
            out.append((t, peak, cap, kv, moved))
            peak = None
    return out
