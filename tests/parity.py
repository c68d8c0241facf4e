"""Parity helpers: compare a GPU decode run with the oracle on the same seeded bytes.

Rules (from the target tolerances), applied per token:
- routing: the selected expert set exact, except where the oracle's k-th and (k+1)-th selection
  scores differ by less than 1e-6 (or, for group-limited routing, the last kept and first dropped
  group scores); such tokens are "exempt" and the pager comparison then follows the GPU's own
  trace.  The rank order inside the set is exact too, except that experts whose oracle scores
  differ by less than 1e-6 may appear in either order (both orders are correct).  At most one token
  in a thousand (at least 2) may be exempt or reordered;
- gates: within 1e-5 of the oracle's gate of the same expert; for exempt tokens, of the oracle's
  gates of the GPU's set;
- pager: hits, misses and fault lists exact against the oracle's Algorithm 1 simulator run on the
  (validated) routing trace;
- outputs: per output row, max |y - o| / max |o| <= 1e-5 (fp32 models) or 2e-2 (bf16 / fp8), where
  o is the oracle's layer, or for exempt tokens the oracle's layer evaluated on the GPU's set.
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
    """Per token.  Returns (exempt, reordered): sets of (step, layer, token).

    A token whose GPU selection equals the oracle's passes.  A token with the same set in another
    rank order passes when that order is valid (scores non-increasing up to NEAR_TIE): "reordered".
    A token whose set differs is "exempt" only at a near-tie: the oracle's k-th and (k+1)-th scores
    within NEAR_TIE, and every expert the GPU chose scores at least the oracle's k-th minus
    NEAR_TIE (it swapped tied candidates, nothing else); or, for group-limited routing, the last
    kept and first dropped group scores within NEAR_TIE.  Every other token must match exactly.
    The outputs and gates of exempt tokens are still checked, against the oracle evaluated on the
    GPU's set (check_gates / check_outputs)."""
    exempt, reordered = set(), set()
    bad = []
    diff = np.any(gpu_idx != ora_idx, axis=-1)
    for s, l, t in zip(*np.nonzero(diff)):
        s, l, t = int(s), int(l), int(t)
        g, o, sc = gpu_idx[s, l, t], ora_idx[s, l, t], scores[s, l, t]
        if set(g.tolist()) == set(o.tolist()) and _valid_order(g, sc):
            reordered.add((s, l, t))
            continue
        kth = sc[o[-1]]
        tie_k = margin[s, l, t] < NEAR_TIE and all(sc[e] >= kth - NEAR_TIE for e in g.tolist())
        tie_group = gmargin[s, l, t] < NEAR_TIE
        if (tie_k or tie_group) and len(set(g.tolist())) == wl.k and _valid_order(g, sc):
            exempt.add((s, l, t))
        else:
            bad.append((s, l, t, g.tolist(), o.tolist(), float(margin[s, l, t])))
    assert not bad, f"{len(bad)} routing mismatches outside near-ties, first: {bad[:3]}"
    return exempt, reordered


def check_gates(run, gpu_idx, gpu_w, ora_idx, ora_g, exempt):
    """The GPU's gates: positive, summing to 1, and equal (1e-5) to the oracle's gate of the same
    expert; for exempt tokens, to the oracle's gates of the GPU's own set.  Returns the worst error."""
    wl = run.wl
    assert np.allclose(gpu_w.sum(-1), 1.0, atol=1e-5) and (gpu_w > 0).all()
    err = 0.0
    S = gpu_idx.shape[0]
    # ranks may differ only by valid reorders, so compare gate by expert id
    for s in range(S):
        for l in range(wl.L):
            same = np.array_equal(gpu_idx[s, l], ora_idx[s, l])
            if same:
                err = max(err, float(np.abs(gpu_w[s, l] - ora_g[s, l]).max()))
                continue
            for t in range(wl.T):
                if (s, l, t) in exempt:
                    want = oracle.route_gates(wl.route, run.wr_host[l], run.x_host[l, s, t], gpu_idx[s, l, t])
                    err = max(err, float(np.abs(gpu_w[s, l, t] - want).max()))
                    continue
                og = dict(zip(ora_idx[s, l, t].tolist(), ora_g[s, l, t].tolist()))
                for e, g in zip(gpu_idx[s, l, t].tolist(), gpu_w[s, l, t].tolist()):
                    err = max(err, abs(g - og[e]))
    assert err < 1e-5, err
    return err


def routing_bound(S, wl):
    """At most this many tokens may be exempt or reordered (one in a thousand, at least 2)."""
    return max(2, S * wl.L * wl.T // 1000)


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


def check_outputs(run, y_gpu, points, ora_idx=None, threads=None, tokens=None, gpu_idx=None, exempt=()):
    """Oracle layer output at the given (step, layer) points (all tokens, or the listed ones);
    returns the worst row-relative error.  Tokens in `exempt` (step, layer, token) are compared with
    the oracle evaluated on the GPU's routed set gpu_idx (a near-tie where both sets are correct)."""
    wl = run.wl
    tol = tolerance(wl)
    worst = 0.0
    worst_el = 0.0
    tok_all = np.arange(wl.T) if tokens is None else np.asarray(tokens)
    for pt in points:
        s, l = pt[0], pt[1]
        tok = tok_all if len(pt) < 3 else np.asarray(pt[2])
        blobs = run.master_ptrs(l)
        shared = run.shared_ptr(l)
        x = np.ascontiguousarray(run.x_host[l, s][tok])
        idx, g, y, _, _ = oracle.moe_layer(wl.route, blobs, run.wr_host[l], x, wl.k, wl.I, wl.w_dtype,
                                           shared, wl.n_groups, wl.topk_groups)
        ex = [i for i, t in enumerate(tok.tolist()) if (s, l, t) in exempt]
        if ex:
            g_ex, y_ex = oracle.moe_layer_routed(wl.route, blobs, run.wr_host[l], x[ex], gpu_idx[s, l][tok[ex]],
                                                 wl.I, wl.w_dtype, shared)
            idx[ex], g[ex], y[ex] = gpu_idx[s, l][tok[ex]], g_ex, y_ex
        if ora_idx is not None:
            keep = np.setdiff1d(np.arange(len(tok)), ex)
            assert np.array_equal(idx[keep], ora_idx[s, l][tok[keep]])
        yg = y_gpu[s, l][tok].astype(np.float64)
        scale = np.abs(y).max(axis=-1)
        row_err = np.abs(yg - y).max(axis=-1) / scale
        el = np.abs(yg - y) / np.maximum(np.abs(y), 1e-6 * scale[:, None])
        worst = max(worst, float(row_err.max()))
        worst_el = max(worst_el, float(el.max()))
        if row_err.max() > tol:
            for i, t in enumerate(tok.tolist()):
                log(f"  step {s} layer {l} token {t}: experts {idx[i].tolist()} gates {np.round(g[i], 4).tolist()} "
                    f"row-relative error {row_err[i]:.3e}{' (exempt: GPU set)' if i in ex else ''}")
        assert row_err.max() <= tol, f"step {s} layer {l}: row-relative error {row_err.max():.3e} > {tol}"
    return worst, worst_el


def exempt_points(exempt):
    """(step, layer, [tokens]) points that cover every exempt token."""
    by = {}
    for s, l, t in sorted(exempt):
        by.setdefault((s, l), []).append(t)
    return [(s, l, ts) for (s, l), ts in sorted(by.items())]


def check_run(run, out, steps, points, tokens=None, cap=None):
    """Routing (per token, near-ties exempt), gates, pager counts against the oracle's Algorithm 1
    on the GPU's trace (when cap is given), and outputs at `points` plus every exempt token.
    Returns (ora_idx, exempt, reordered, worst, worst_el)."""
    wl = run.wl
    ora_idx, ora_g, margin, gmargin, scores = oracle_routing(run, steps)
    exempt, reordered = check_routing(wl, out["idx"], ora_idx, margin, gmargin, scores)
    assert len(exempt) + len(reordered) <= routing_bound(steps, wl), (len(exempt), len(reordered))
    check_gates(run, out["idx"], out["w"], ora_idx, ora_g, exempt)
    if cap is not None:
        check_pager(wl, cap, out["idx"], out["hits"], out["misses"], out.get("chunks"))
    worst, worst_el = check_outputs(run, out["y"], points, ora_idx, tokens=tokens, gpu_idx=out["idx"],
                                    exempt=exempt)
    if exempt:
        check_outputs(run, out["y"], exempt_points(exempt), ora_idx, gpu_idx=out["idx"], exempt=exempt)
    return ora_idx, exempt, reordered, worst, worst_el


def check_masters_unchanged(run, pairs):
    """The master blobs of the (layer, expert) pairs still hold what the seeded generator wrote
    (expert -1: the shared expert).  Reports the first differing 8-byte words of any that changed."""
    from paper_2606_21868_amd import datagen as dg
    wl = run.wl
    changed = []
    for l, e in sorted(set(pairs)):
        got = run.master_blob(l, e)
        want = dg.expert_blob(wl.seed, l, dg.SHARED_EXPERT if e < 0 else e, wl.w_dtype, wl.d, wl.I)[:got.size]
        ne = np.flatnonzero(got != want)
        if ne.size:
            w0 = int(ne[0]) & ~7
            changed.append((l, e, int(ne.size), int(ne[0]), int(ne[-1]), got[w0:w0 + 32].tobytes().hex(),
                            want[w0:w0 + 32].tobytes().hex()))
    for c in changed[:8]:
        log(f"  master of layer {c[0]} expert {c[1]} changed: {c[2]} bytes in [{c[3]}, {c[4]}]; at the first: "
            f"{c[5]} (generator: {c[6]})")
    return changed


def check_slots_hold_masters(run, max_bytes=4e9):
    """Every resident slot holds its expert's master bytes (all slots when their bytes are at most
    max_bytes, else 32 slots spread over the layers); returns the number checked."""
    wl, cap = run.wl, run.ctx.cap()
    pairs = [(l, s) for l in range(wl.L) for s in range(cap)]
    if len(pairs) * run.blob_bytes > max_bytes:
        pairs = [pairs[i] for i in np.linspace(0, len(pairs) - 1, 32).astype(int)]
    n = 0
    for l, s in pairs:
        e = run.ctx.expert_in_slot(l, s)
        if e < 0:
            continue
        got, want = run.ctx.read_slot(l, s, run.blob_bytes), run.master_blob(l, e)
        ne = np.flatnonzero(got != want)
        assert ne.size == 0, (f"layer {l} slot {s} expert {e}: {ne.size} bytes differ from the master "
                              f"(first {int(ne[0])}, last {int(ne[-1])})")
        n += 1
    return n


def run_case(wl, cap, steps, sample_points=None, check_all_outputs=False, tokens=None, expect_grouped=None,
             pageable=False):
    """Paged run from a cold table, checked against the oracle (routing, pager, outputs at all or the
    sampled (step, layer) points, optionally on a subset of tokens); the device pager where it
    applies; then the fully resident run (C = N, preloaded) must give bit-identical outputs."""
    import pytest

    from paper_2606_21868_amd import wisp
    log(f"[case] {wl.name} L={wl.L} d={wl.d} I={wl.I} N={wl.N} k={wl.k} T={wl.T} steps={steps} C={cap}"
        f"{' (pageable masters)' if pageable else ''}")
    run = wisp.DecodeRun(wl, device=0, steps=steps, pageable=pageable)
    try:
        run.generate()
        log(f"  generated in {run.gen_seconds:.1f}s; paged decode from cold")
        assert run.set_cap(cap) == cap
        if expect_grouped is not None:
            run.ctx.set_profiling((1 << wisp.K_GROUPED_GATEUP) | (1 << wisp.K_FFN_GATEUP))
        out = run.decode(record=True)
        if expect_grouped is not None:
            run.ctx.set_profiling(0)
            n_grouped = run.ctx.kernel_times(wisp.K_GROUPED_GATEUP)["launches"]
            n_items = run.ctx.kernel_times(wisp.K_FFN_GATEUP)["launches"]
            assert (n_grouped > 0, n_items > 0) == (expect_grouped, not expect_grouped), (n_grouped, n_items)
            log(f"  expert FFN path: {'grouped MFMA GEMMs' if expect_grouped else 'per-item GEMV'} "
                f"({n_grouped + n_items} gate/up launches)")
        log("  oracle routing")
        ora_idx, ora_g, margin, gmargin, scores = oracle_routing(run, steps)
        exempt, reordered = check_routing(wl, out["idx"], ora_idx, margin, gmargin, scores)
        log(f"  routing ok ({len(exempt)} near-tie tokens exempt, {len(reordered)} with near-equal ranks "
            f"swapped); pager vs Algorithm 1 simulator")
        assert len(exempt) + len(reordered) <= routing_bound(steps, wl)
        check_pager(wl, cap, out["idx"], out["hits"], out["misses"], out["chunks"])
        check_gates(run, out["idx"], out["w"], ora_idx, ora_g, exempt)
        if check_all_outputs:
            points = [(s, l) for s in range(steps) for l in range(wl.L)]
        else:
            points = list(sample_points)
        # every exempt token is checked too (against the oracle on the GPU's set), also outside the sample
        if not check_all_outputs or tokens is not None:
            points += [p for p in exempt_points(exempt)]
        log(f"  outputs at {len(points)} (step, layer) points")
        if pageable:
            # the oracle reads the masters now, long after the fills copied them: check that they
            # still hold the generator's bytes (up to 16 blobs used at the checked points)
            first = sorted({(points[0][1], int(e)) for e in np.unique(out["idx"][points[0][:2]])})
            rest = sorted({(p[1], int(e)) for p in points for e in np.unique(out["idx"][p[0], p[1]])} - set(first))
            if wl.has_shared:
                rest += sorted({(p[1], -1) for p in points})
            n_rest = min(len(rest), max(0, 16 - len(first)))
            used = first + [rest[i] for i in np.linspace(0, len(rest) - 1, n_rest).astype(int)] if n_rest else first
            changed = check_masters_unchanged(run, used)
            assert not changed, f"{len(changed)} pageable master blobs changed during the run"
            log(f"  {len(used)} master blobs used at the checked points unchanged since generation")
        try:
            worst, worst_el = check_outputs(run, out["y"], points, ora_idx, tokens=tokens, gpu_idx=out["idx"],
                                            exempt=exempt)
        except AssertionError:
            # replay the same steps from cold: a transient error (ordering) gives different bits, a
            # reproducible one the same
            run.ctx.masters_ready()
            again = run.decode(record=True)
            same = np.array_equal(again["y"].view(np.uint32), out["y"].view(np.uint32))
            log(f"  replay from cold: outputs {'bit-identical to' if same else 'differ from'} the first run")
            try:
                check_outputs(run, again["y"], points, ora_idx, tokens=tokens, gpu_idx=out["idx"], exempt=exempt)
                log("  replay: every point within tolerance")
            except AssertionError as e2:
                log(f"  replay also fails: {e2}")
            raise
        log(f"  worst row-relative error {worst:.3e} (elementwise {worst_el:.3e}); total misses "
            f"{int(out['misses'].sum())} of {int(out['hits'].sum() + out['misses'].sum())} references")
        n_slots = check_slots_hold_masters(run)
        log(f"  {n_slots} resident slots byte-equal to their masters")
        tables = [[run.ctx.slot_of(l, e) for e in range(wl.N)] for l in range(wl.L)]
        # the device pager: same trace from cold -> same decisions, same slots, same bits
        device_ok = cap >= wl.T * wl.k and wl.T <= 4 and not pageable
        run.ctx.masters_ready()            # drops every resident expert
        run.ctx.reset_stats()
        if device_ok:
            try:
                run.ctx.set_pager(wisp.PAGER_DEVICE)
            except wisp.WispError as e:   # a layer shape the device-planned kernels do not cover
                assert e.status == wisp.E_INVAL and "not supported" in str(e), e
                device_ok = False
        if device_ok:
            dev = run.decode(record=True)
            assert np.array_equal(dev["idx"], out["idx"])
            assert np.array_equal(dev["hits"], out["hits"]) and np.array_equal(dev["misses"], out["misses"])
            assert [[run.ctx.slot_of(l, e) for e in range(wl.N)] for l in range(wl.L)] == tables
            assert np.array_equal(dev["y"].view(np.uint32), out["y"].view(np.uint32)), "device pager changed bits"
            # the device pager's gate/up launch fills the faulted slots itself (W1/W3 while computing, the
            # rest of the blob by workgroups of its own)
            n_dev = check_slots_hold_masters(run)
            log(f"  device pager: same routing, faults, slot tables and output bits as the host pager; {n_dev} "
                f"resident slots byte-equal to their masters")
        elif not (cap >= wl.T * wl.k and wl.T <= 4 and not pageable):
            with pytest.raises(wisp.WispError) as ei:
                run.ctx.set_pager(wisp.PAGER_DEVICE)
            assert ei.value.status == wisp.E_INVAL
        # fully resident: C = N, preloaded, same kernels -> bit-identical, no faults
        assert run.set_cap(wl.N) == wl.N
        run.ctx.preload()
        run.ctx.reset_stats()
        res = run.decode(record=True)
        assert int(res["misses"].sum()) == 0
        assert np.array_equal(res["idx"], out["idx"])
        assert np.array_equal(res["y"].view(np.uint32), out["y"].view(np.uint32)), "paged != resident bits"
        log(f"  paged output bit-identical to the fully resident run ({'device' if device_ok else 'host'} pager)")
        return out
    finally:
        run.close()


def check_prediction(ids, scores, exact, depth):
    """ids/scores from the library against the oracle's exact scores: every score within 1e-12
    (relative), the order non-increasing with ties in id order, and the set equal to the oracle's
    top `depth` up to candidates tied with the last kept score."""
    assert len(ids) == len(scores)
    for e, s in zip(ids, scores):
        assert abs(s - float(exact[e])) <= 1e-12 * max(1.0, float(exact[e])), (e, s, exact[e])
    for a, b in zip(ids[:-1], ids[1:]):
        assert exact[a] > exact[b] or (exact[a] == exact[b] and a < b) or abs(float(exact[a] - exact[b])) < 1e-12
    positive = sorted((e for e in range(len(exact)) if exact[e] > 0), key=lambda e: (-exact[e], e))
    assert len(ids) == min(depth, len(positive))
    if ids:
        cut = exact[ids[-1]]
        above = {e for e in positive if exact[e] > cut and float(exact[e] - cut) >= 1e-12}
        assert above <= set(ids)
