"""Parity helpers: compare a GPU decode run with the oracle on the same seeded bytes.

Rules (from the target tolerances):
- routing: the selected expert set exact, except where the oracle's k-th and (k+1)-th selection
  scores differ by less than 1e-6 (or, for group-limited routing, the last kept and first dropped
  group scores); such layer-steps are "exempt" and the pager comparison then follows the GPU's
  own trace.  The rank order inside the set is exact too, except that experts whose oracle
  scores differ by less than 1e-6 may appear in either order (both orders are correct);
- pager: hits, misses and fault lists exact against the oracle's Algorithm 1 simulator run on the
  (validated) routing trace;
- outputs: per output row, max |y - o| / max |o| <= 1e-5 (fp32 models) or 2e-2 (bf16 / fp8).
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import sys

import numpy as np

import oracle

NEAR_TIE = 1e-6


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def tolerance(wl):
    return 1e-5 if wl.w_dtype == oracle.F32 else 2e-2


def oracle_routing(run, steps=None, threads=None):
    """Oracle routing of every (step, layer, token): idx [S,L,T,k], gates, margins [S,L,T], group margins."""
    wl = run.wl
    S = steps if steps is not None else run.x_host.shape[1]
    idx = np.zeros((S, wl.L, wl.T, wl.k), np.int32)
    gates = np.zeros((S, wl.L, wl.T, wl.k), np.float64)
    margin = np.zeros((S, wl.L, wl.T), np.float64)
    gmargin = np.full((S, wl.L, wl.T), np.inf)
    scores = np.zeros((S, wl.L, wl.T, wl.N), np.float64)

    def one(args):
        s, l = args
        for t in range(wl.T):
            i, g, sc, m, gm = oracle.route(wl.route, run.wr_host[l], run.x_host[l, s, t], wl.k, wl.n_groups,
                                           wl.topk_groups)
            idx[s, l, t], gates[s, l, t], margin[s, l, t], gmargin[s, l, t], scores[s, l, t] = i, g, m, gm, sc

    jobs = [(s, l) for s in range(S) for l in range(wl.L)]
    with cf.ThreadPoolExecutor(max_workers=threads or min(16, os.cpu_count() or 4)) as ex:
        list(ex.map(one, jobs))
    return idx, gates, margin, gmargin, scores


def _valid_order(gpu_row, scores_row):
    """The GPU's rank order is a correct order of its set: scores non-increasing up to ties below
    the near-tie tolerance, and equal scores in ascending id."""
    for a, b in zip(gpu_row[:-1], gpu_row[1:]):
        sa, sb = scores_row[a], scores_row[b]
        if sa < sb - NEAR_TIE:
            return False
        if sa == sb and a > b:
            return False
    return True


def check_routing(wl, gpu_idx, ora_idx, margin, gmargin, scores):
    """Returns (exempt, reordered): layer-steps whose selected set differs at a near-tie boundary,
    and layer-steps whose set matches but whose rank order differs among near-equal scores.
    Asserts exact agreement everywhere else."""
    S = ora_idx.shape[0]
    exempt, reordered = set(), set()
    bad = []
    for s in range(S):
        for l in range(wl.L):
            if np.array_equal(gpu_idx[s, l], ora_idx[s, l]):
                continue
            same_sets = all(set(gpu_idx[s, l, t].tolist()) == set(ora_idx[s, l, t].tolist()) for t in range(wl.T))
            if same_sets and all(_valid_order(gpu_idx[s, l, t], scores[s, l, t]) for t in range(wl.T)):
                reordered.add((s, l))
                continue
            near = bool(np.any(margin[s, l] < NEAR_TIE) or np.any(gmargin[s, l] < NEAR_TIE))
            if near:
                exempt.add((s, l))
            else:
                bad.append((s, l, gpu_idx[s, l].tolist(), ora_idx[s, l].tolist(), margin[s, l].tolist()))
    assert not bad, f"{len(bad)} routing mismatches outside near-ties, first: {bad[:3]}"
    return exempt, reordered


def check_pager(wl, cap, gpu_idx, hits, misses, chunks=None):
    """Run the oracle's Algorithm 1 simulator per layer over the GPU's routing trace and compare."""
    S = gpu_idx.shape[0]
    for l in range(wl.L):
        sim = oracle.LRU(wl.N, cap)
        for s in range(S):
            r = sim.step(gpu_idx[s, l].ravel())
            got = (int(hits[s, l]), int(misses[s, l]))
            assert got == (r["hits"], r["misses"]), f"layer {l} step {s}: gpu {got} oracle {(r['hits'], r['misses'])}"
            if chunks is not None:
                assert int(chunks[s, l]) == r["chunks"], f"layer {l} step {s}: chunks"
    return True


def check_outputs(run, y_gpu, points, ora_idx=None, threads=None):
    """Oracle layer output at the given (step, layer) points; returns the worst row-relative error."""
    wl = run.wl
    tol = tolerance(wl)
    worst = 0.0
    worst_el = 0.0
    for (s, l) in points:
        blobs = run.master_ptrs(l)
        shared = run.shared_ptr(l)
        idx, g, y, _, _ = oracle.moe_layer(wl.route, blobs, run.wr_host[l], run.x_host[l, s], wl.k, wl.I, wl.w_dtype,
                                           shared, wl.n_groups, wl.topk_groups)
        if ora_idx is not None:
            assert np.array_equal(idx, ora_idx[s, l])
        yg = y_gpu[s, l].astype(np.float64)
        scale = np.abs(y).max(axis=-1)
        row_err = np.abs(yg - y).max(axis=-1) / scale
        el = np.abs(yg - y) / np.maximum(np.abs(y), 1e-6 * scale[:, None])
        worst = max(worst, float(row_err.max()))
        worst_el = max(worst_el, float(el.max()))
        assert row_err.max() <= tol, f"step {s} layer {l}: row-relative error {row_err.max():.3e} > {tol}"
    return worst, worst_el
