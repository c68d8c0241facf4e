#!/usr/bin/env python3
"""Benchmark: paged MoE decode tokens/s at a fixed VRAM expert budget, one MI355X.

Workload (default): Qwen3-30B-A3B-shaped paged decode — 48 MoE layers, d=2048, 128 bf16 experts
per layer (SwiGLU, I=768, 9,437,184-byte blobs), top-8 softmax-then-renormalise routing, batch 1,
AR(1) hidden states, expert budget 25% of the 6144 experts (C = 32 slots per layer), LRU paging
from pinned host masters.  A step is one decode token through all 48 layers: router + top-k,
slot lookup and fault list, host->device fills of the faults, slot-indirected SwiGLU FFN and
combine, layer after layer.  Inputs (weights in pinned host memory, hidden states in HBM) are in
place before the timed region; every step starts from the slot contents the previous one left.

Reported beside the throughput:
  roofline       the expert gate/up GEMV kernel (the largest share of HBM bytes): algorithmic
                 bytes per launch / average launch time from HIP events over the timed region,
                 against the 8 TB/s HBM peak;
  path_roofline  the whole path against T_roof = sum over layer-steps of HBM bytes / 8 TB/s +
                 fault bytes / measured host-link bandwidth of the engine that moves them (compute-unit
                 streaming for the device pager, the copy engine for the host pager; exact fault counts
                 of the run);
  cpu_baseline   the fp64 CPU oracle (fully resident layer) on a bounded sample of the same
                 workload, on this host's cores;
  sweep          at per-layer caps 8..128, the pager against static layer-level offload at the same VRAM
                 expert budget: zero-copy (the routed experts of non-resident layers read over the link
                 each step; the paper-analogue comparison) and bulk (the rest copied whole each step);
  controller     the online dual-resize (Sec. 3.5, App. B) over a KV-occupancy trace with regime
                 shifts: moves made at drained barriers, decode tokens/s per regime against the fixed
                 split;
  configurator   MV-WSA's startup split (Eqs. 3-5) from the miss curve of the GPU's own routing trace,
                 run and compared with the curve's fault prediction;
  prefetch       speculative prefetch (Sec. 4) at caps 8/16/32: off, the online co-activation predictor
                 (App. E), and perfect hints (each step's true routing), on the host pager;
  prefill        the Qwen3-30B-A3B-shaped prefill chunk (2048 tokens per layer, same weights and
                 cap): tokens/s of a cold pass against T_roof = fault bytes / link + max(HBM bytes /
                 8 TB/s, FLOPs / 2.5 PFLOP/s), and the matrix-core rate of the grouped GEMMs in a
                 fully resident pass.
Usage: python bench.py [--gpus 1] [--steps K] [--warmup W]
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
PINNED_LIMIT_BYTES = 60e9           # pinned host memory one process may hold on the test machines (65 GiB)
MFMA_BF16_PEAK_TFLOPS = 2500.0      # dense bf16 matrix-core peak of the MI355X
PREFILL_WORKLOAD = "qwen3-30b-a3b-prefill"
# committed PMC traffic summaries of a kernel class on a workload (their source hash must still match)
TRAFFIC_SUMMARIES = {
    ("qwen3-30b-a3b-decode", "ffn_gateup"): os.path.join(ROOT, "profiles", "ffn_gateup_qwen3-30b-a3b-decode_hbm_traffic.txt"),
    ("deepseek-v3-16l-decode", "ffn_gateup"): os.path.join(ROOT, "profiles",
                                                           "ffn_gateup_fp8_deepseek-v3-16l-decode_profile.txt"),
}
FFN_SOURCE = os.path.join(ROOT, "paper_2606_21868_amd", "csrc", "expert_ffn.hip")


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def measure_hbm_copy(torch, wisp, nbytes=1 << 30, reps=5):
    src = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    s = torch.cuda.Stream()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    rates = []
    with torch.cuda.stream(s):
        wisp.hbm_copy(src, dst, nbytes, s)
        for _ in range(reps):
            ev0.record(s)
            wisp.hbm_copy(src, dst, nbytes, s)
            ev1.record(s)
            ev1.synchronize()
            rates.append(2 * nbytes / (ev0.elapsed_time(ev1) * 1e-3) / 1e9)
    del src, dst
    rates.sort()
    return rates[len(rates) // 2]


def measured_traffic(workload, kname):
    """HBM bytes per launch of kernel class kname from its committed FETCH_SIZE/WRITE_SIZE counter summary
    (scaled by the copy-kernel calibration it records), or None when there is none for this workload and
    kernel or the kernel source has changed since the counters were taken."""
    import hashlib
    summary = TRAFFIC_SUMMARIES.get((workload, kname))
    if summary is None or not os.path.exists(summary):
        return None
    fields = {}
    for line in open(summary):
        parts = line.split()
        if len(parts) >= 2 and parts[0].startswith("traffic_"):
            fields[parts[0]] = float(parts[1])
        elif parts[:2] == ["kernel_source", "expert_ffn.hip"] and len(parts) == 4:
            fields["sha256"] = parts[3]
    with open(FFN_SOURCE, "rb") as f:
        if hashlib.sha256(f.read()).hexdigest() != fields.get("sha256"):
            return None
    if "traffic_bytes_per_launch" not in fields:
        return None
    return dict(bytes_per_launch=fields["traffic_bytes_per_launch"],
                algorithmic_bytes_per_launch=fields.get("traffic_algorithmic_bytes_per_launch"),
                source=os.path.relpath(summary, ROOT))


def cpu_baseline(run, wl, start_step, max_tokens=24, budget_s=15.0):
    """The oracle as it stands: fully resident fp64 layer, layer after layer of consecutive decode
    steps, until max_tokens tokens or the time budget; a partial step counts its share of layers."""
    import oracle
    threads = oracle.num_threads()
    t0 = time.perf_counter()
    layers = 0
    s = start_step
    while layers < max_tokens // wl.T * wl.L and s < run.x_host.shape[1]:
        l = layers % wl.L
        oracle.moe_layer(wl.route, run.master_ptrs(l), run.wr_host[l], run.x_host[l, s], wl.k, wl.I, wl.w_dtype,
                         run.shared_ptr(l), wl.n_groups, wl.topk_groups)
        layers += 1
        if layers % wl.L == 0:
            s += 1
        if time.perf_counter() - t0 > budget_s:
            break
    dt = time.perf_counter() - t0
    tokens = layers / wl.L * wl.T
    return dict(value=tokens / dt, unit="tokens/s", cores=threads, kind="oracle",
                sample=f"{layers} layer-steps ({layers / wl.L:.2f} decode steps of {wl.L} layers) x batch {wl.T} "
                       f"(fully resident fp64 layer, weights read from the same host masters), {dt:.1f} s")


SWEEP_CAPS = (8, 16, 32, 64, 128)


def sweep_leg(run, wl, wisp, torch, warmup=16, steps=96, offload_steps=3):
    """Iso-VRAM sweep over the expert budget (the analogue of the paper's Fig. 3 and Table 1): at each
    per-layer cap C the budget is C * L * M_e bytes, spent three ways on the same steps and kernels:
    the pager (device pager, cold start; preloaded when C = N, where every expert fits), zero-copy
    offload (whole layers resident, the routed experts of the other layers read over the host link each
    step, nothing cached: the bytes per token the paper's measured static-offload rates imply, so the
    paper-analogue comparison), and bulk offload (whole layers resident, every other layer copied in
    bulk each step: the layer-grained reading of the baseline, a lower bound)."""
    steps = min(steps, run.steps - warmup)
    out = []

    def timed(fn, n):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        fn(n)
        torch.cuda.synchronize()
        return wl.T * n / (time.perf_counter() - t0)

    for cap in SWEEP_CAPS:
        if cap > wl.N:
            continue
        budget = cap * wl.L * wl.blob
        run.ctx.set_pager(wisp.PAGER_HOST)
        run.ctx.masters_ready()
        assert run.set_cap(cap) == cap
        if cap == wl.N:
            run.ctx.preload()
        run.ctx.set_pager(wisp.PAGER_DEVICE)
        run.decode(record=False, steps=warmup, start=0, stats=False)
        faults = {}

        def paged_run(n):
            faults["n"] = int(run.decode(record=False, steps=n, start=warmup)["misses"].sum())

        paged = timed(paged_run, steps)
        resident = resident_roofline(run, wl, wisp, paged, warmup) if cap == wl.N else None
        run.ctx.set_pager(wisp.PAGER_HOST)
        arms = {}
        for mode, name in ((wisp.OFFLOAD_BULK, "static_offload"), (wisp.OFFLOAD_ZERO_COPY, "zero_copy_offload")):
            r = run.ctx.offload_begin(budget, mode)
            run.offload(record=False, steps=1, start=0)
            n = offload_steps if (mode == wisp.OFFLOAD_BULK and r < wl.L) else 4 * offload_steps
            arms[name] = (timed(lambda n: run.offload(record=False, steps=n, start=1), n), r)
            run.ctx.offload_end()
        st, zc = arms["static_offload"], arms["zero_copy_offload"]
        out.append(dict(cap=cap, budget_GB=budget / 1e9, paged_tokens_per_s=paged, paged_preloaded=cap == wl.N,
                        paged_faults_per_token=faults["n"] / (wl.T * steps),
                        zero_copy_offload_tokens_per_s=zc[0], zero_copy_resident_layers=zc[1],
                        speedup_vs_zero_copy=paged / zc[0],
                        bulk_offload_tokens_per_s=st[0], bulk_resident_layers=st[1],
                        speedup_vs_bulk=paged / st[0]))
        if resident:
            out[-1]["resident"] = resident
        log(f"sweep C={cap:3d} ({budget / 1e9:5.1f} GB): paged {paged:7.2f} tokens/s; zero-copy offload {zc[0]:7.2f} "
            f"({zc[1]} resident layers) -> {paged / zc[0]:4.1f}x; bulk offload {st[0]:7.2f} ({st[1]}) -> "
            f"{paged / st[0]:5.1f}x")
    return out


def resident_roofline(run, wl, wisp, tokens_per_s, start, census_steps=24):
    """Every expert resident (C = N, preloaded, device pager): the decode path is HBM-bound, with
    T_roof = (k experts' blobs + the fp32 router matrix) per layer / 8 TB/s.  Reports that fraction and,
    from census steps with every kernel class event-timed, each kernel's launch time and HBM rate
    (algorithmic bytes: the router matrix for the fused router + selection + paging kernel, the k
    experts' W1/W3 rows for gate/up, their W2 rows for down + combine)."""
    hbm_per_token = wl.L * (wl.T * wl.k * wl.blob + wl.N * wl.d * 4)
    roof = HBM_PEAK_GBPS * 1e9 / hbm_per_token * wl.T
    run.ctx.reset_kernel_times()
    run.ctx.set_profiling(True)
    run.decode(record=False, steps=census_steps, start=start, stats=False)
    run.ctx.set_profiling(0)
    wbytes = 2 if wl.w_dtype == wisp.BF16 else 4
    per_launch = {"router_select": wl.N * wl.d * 4, "ffn_gateup": wl.T * wl.k * 2 * wl.d * wl.I * wbytes,
                  "down_combine": wl.T * wl.k * wl.d * wl.I * wbytes}
    kern = {}
    for kc, name in enumerate(wisp.KERNEL_CLASS_NAMES):
        t = run.ctx.kernel_times(kc)
        if not t["launches"]:
            continue
        avg_us = t["total_ms"] * 1e3 / t["launches"]
        e = dict(launches=t["launches"], avg_us=avg_us)
        if name in per_launch:
            gbps = per_launch[name] / (avg_us * 1e-6) / 1e9
            e.update(bytes_per_launch=per_launch[name], GBps=gbps, frac_of_hbm_peak=gbps / HBM_PEAK_GBPS)
        kern["route_page" if name == "router_select" else name] = e
    log(f"resident decode (C = N): {tokens_per_s:.0f} tokens/s = {tokens_per_s / roof:.3f} of its HBM roofline "
        f"({roof:.0f}); " + ", ".join(f"{k} {v['avg_us']:.2f} us" + (f" ({v['frac_of_hbm_peak']:.2f} of HBM)"
                                                                    if 'frac_of_hbm_peak' in v else "")
                                      for k, v in kern.items()))
    return dict(hbm_bytes_per_token=hbm_per_token, roofline_tokens_per_s=roof, frac=tokens_per_s / roof,
                us_per_layer_step=1e6 / tokens_per_s * wl.T / wl.L, kernels=kern,
                kernel_source="census steps after the timed ones, every kernel class event-timed")


def configurator_leg(run, wl, wisp, torch, link_cu, warmup=16, steps=96):
    """MV-WSA's startup configurator (Sec. 3.3-3.4, Eqs. 3-5) fed by the GPU's own routing.  The expert
    miss curve m_exp(C) is the sum over layers of the library's reuse-distance curve of the routing the
    pager recorded over the whole run (with its upper bound beside it); the KV side is a stand-in: a
    demand of D blocks, each block short of
    it recomputed every step (m_kv = max(0, demand - kappa), c_kv = KV_RECOMPUTE_S per block), with the
    admission floor of Eq. 4 for four sessions of 4096 tokens.  c_exp = M_e / the measured compute-unit
    link rate.  The KV demand is the peak of the occupancy model's tool-call regime (the representative
    trace of the offline mode).  The chosen split is then run (device pager, cold) and its faults
    compared with the curve's prediction."""
    import numpy as np

    from paper_2606_21868_amd.workloads import kv_occupancy_trace
    a = wl.L * wl.blob
    b = KV_BLOCK_BYTES
    kv0 = int(KV_POOL_GIB * (1 << 30)) // b
    B = wl.cap * a + kv0 * b
    demand = int(kv_occupancy_trace([(160, "tool")], kv0, seed=0).max())
    run.ctx.set_pager(wisp.PAGER_HOST)
    run.ctx.masters_ready()
    assert run.set_cap(wl.cap) == wl.cap
    run.ctx.set_pager(wisp.PAGER_DEVICE)
    rec = run.decode(record=True, steps=run.steps, start=0)
    S = run.steps

    def curves(n_steps):
        """Sum over layers of the lower and upper curves of the first n_steps of the recorded routing."""
        lo_, up_ = np.zeros(wl.N + 1), np.zeros(wl.N + 1)
        for l in range(wl.L):
            c_lo, c_up = wisp.miss_curve(rec["idx"][:n_steps, l].reshape(n_steps, -1), wl.N, upper=True)
            lo_ += c_lo
            up_ += c_up
        return lo_, up_

    lo, up = curves(S)
    # a reference's classification depends only on earlier steps, so the faults of the window the
    # chosen split is timed on are the curves of the longer prefix minus those of the warmup prefix
    lo_w, up_w = [a - b for a, b in zip(curves(warmup + steps), curves(warmup))]
    lo_warm, _ = curves(warmup)
    m_exp = np.round((lo - lo_warm) / (S - warmup)).astype(np.uint64)   # expert faults per warm decode step
    kv_min = 4 * math.ceil(4096 / 16)
    m_kv = np.maximum(0, demand - np.arange(demand + 1)).astype(np.float64)
    c_exp = wl.blob / (link_cu * 1e9)
    split = wisp.mvwsa_configure(B, a, b, kv_min, c_exp, KV_RECOMPUTE_S, m_exp, m_kv)
    cap = split["cap"]
    run.ctx.set_pager(wisp.PAGER_HOST)
    run.ctx.masters_ready()
    assert run.set_cap(cap) == cap
    run.ctx.set_pager(wisp.PAGER_DEVICE)
    run.decode(record=False, steps=warmup, start=0, stats=False)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    o = run.decode(record=False, steps=steps, start=warmup)
    torch.cuda.synchronize()
    el = time.perf_counter() - t0
    run.ctx.set_pager(wisp.PAGER_HOST)
    assert run.set_cap(wl.cap) == wl.cap
    whole = rec["misses"].sum()
    res = dict(budget_GiB=B / (1 << 30), kv_block_bytes=b, kv_demand_blocks=demand, kv_min_blocks=kv_min,
               c_exp_s=c_exp, c_kv_s=KV_RECOMPUTE_S, split=split, kv_GiB=split["kv_blocks"] * b / (1 << 30),
               curve_faults_per_step=dict(C={int(c): [float(lo[c] / S), float(up[c] / S)]
                                             for c in (8, 16, 32, 64, 128, cap) if c <= wl.N}),
               recorded_cap=wl.cap, recorded_faults_per_step=float(whole / S),
               recorded_within_curves=bool(lo[wl.cap] <= whole <= up[wl.cap]),
               chosen=dict(cap=cap, tokens_per_s=wl.T * steps / el, window_steps=[warmup, warmup + steps],
                           faults_per_step=float(o["misses"].sum()) / steps,
                           curve_bounds_per_step=[float(lo_w[cap] / steps), float(up_w[cap] / steps)],
                           within_curves=bool(lo_w[cap] <= o["misses"].sum() <= up_w[cap])))
    log(f"configurator: B {B / (1 << 30):.2f} GiB -> cap {cap} / KV {res['kv_GiB']:.2f} GiB (f = {split['f']:.3f}, "
        f"floor binding {split['floor_binding']}); decode {res['chosen']['tokens_per_s']:.2f} tokens/s, "
        f"{res['chosen']['faults_per_step']:.1f} faults per step (curve {lo_w[cap] / steps:.1f}..{up_w[cap] / steps:.1f})")
    return res


# Qwen3-30B-A3B KV cache: 48 layers x (K, V) x 4 KV heads x 128 x bf16 per token, 16-token blocks
KV_BLOCK_BYTES = 16 * 48 * 2 * 4 * 128 * 2
KV_POOL_GIB = 2.79          # the fixed split's KV pool in the paper's live run
KV_HEADROOM = 0.2
KV_DEAD_ZONE = 2            # experts per layer
KV_RECOMPUTE_S = 16 / 91000.0   # recomputing one 16-token block at the resident prefill rate
CONTROLLER_BARRIER_EVERY = 32
CONTROLLER_REGIMES = (("tool", 160), ("long", 160), ("tool", 160))


def controller_leg(run, wl, wisp, torch, warmup=16):
    """The online dual-resize of Sec. 3.5 / App. B on the decode workload (device pager).  A seeded
    KV-occupancy trace with regime shifts (four sessions; short tool-call bursts, then long-context
    turns, then bursts again) is observed step by step; every CONTROLLER_BARRIER_EVERY steps, at a
    drained barrier, the controller takes the peak since the last barrier and applies the control law
    (Eqs. 6-8, headroom KV_HEADROOM, dead-zone KV_DEAD_ZONE) to the expert scratch and a KV pool of real
    device memory (the KV cache itself is simulated: its bytes are held, not read).  The same steps run
    on the fixed split (cap 32, 2.79 GiB of KV).  Per regime: decode tokens/s of both, and the steps
    whose occupancy exceeded the pool in place (requests that would be preempted)."""
    import numpy as np

    from paper_2606_21868_amd.workloads import kv_occupancy_trace
    a = wl.L * wl.blob
    b = KV_BLOCK_BYTES
    kv0 = int(KV_POOL_GIB * (1 << 30)) // b
    B = wl.cap * a + kv0 * b
    every = CONTROLLER_BARRIER_EVERY
    steps = sum(n for _, n in CONTROLLER_REGIMES)
    steps = min(steps, (run.steps - warmup) // every * every)
    occ = kv_occupancy_trace([(n, k) for k, n in CONTROLLER_REGIMES], kv0, seed=0)[:steps]
    regime = np.concatenate([[k] * n for k, n in CONTROLLER_REGIMES])[:steps]

    def pass_(live):
        run.ctx.set_pager(wisp.PAGER_HOST)
        assert run.set_cap(wl.cap) == wl.cap
        run.ctx.masters_ready()
        pool = wisp.KvPool(b, kv0)
        ctl = wisp.Controller(B, a, b, 0, KV_HEADROOM, 1, wl.N, KV_DEAD_ZONE, wl.cap, kv0) if live else None
        try:
            run.ctx.set_pager(wisp.PAGER_DEVICE)
            run.decode(record=False, steps=warmup, start=0, stats=False)
            win_s, moves, over = [], [], np.zeros(steps, bool)
            for s0 in range(0, steps, every):
                kv_now = pool.blocks
                torch.cuda.synchronize()
                t0 = time.perf_counter()
                run.decode(record=False, steps=every, start=warmup + s0, stats=False)
                torch.cuda.synchronize()
                win_s.append(time.perf_counter() - t0)
                over[s0:s0 + every] = occ[s0:s0 + every] > kv_now
                if ctl is not None:
                    for t in range(s0, s0 + every):
                        ctl.observe(int(occ[t]))
                    t1 = time.perf_counter()
                    cap, kv, moved, peak = ctl.barrier(run.ctx, pool)       # drains, then moves
                    dt = time.perf_counter() - t1
                    if moved:
                        moves.append(dict(step=s0 + every, peak_blocks=peak, cap=cap, kv_GiB=kv * b / (1 << 30),
                                          moved=moved, seconds=dt))
            per = {}
            for k, _ in CONTROLLER_REGIMES:
                idx = [i for i in range(len(win_s)) if regime[i * every] == k]
                per[k] = dict(tokens_per_s=wl.T * every * len(idx) / sum(win_s[i] for i in idx),
                              steps_over_pool=int(sum(over[i * every:(i + 1) * every].sum() for i in idx)))
            return dict(tokens_per_s=wl.T * steps / sum(win_s), per_regime=per, moves=moves,
                        final_cap=run.ctx.cap(), final_kv_GiB=pool.blocks * b / (1 << 30))
        finally:
            if ctl is not None:
                ctl.close()
            pool.close()

    fixed = pass_(False)
    live = pass_(True)
    run.ctx.set_pager(wisp.PAGER_HOST)
    assert run.set_cap(wl.cap) == wl.cap
    res = dict(budget_GiB=B / (1 << 30), kv_block_bytes=b, barrier_every=every, headroom=KV_HEADROOM,
               dead_zone=KV_DEAD_ZONE, regimes=[dict(kind=k, steps=n) for k, n in CONTROLLER_REGIMES],
               fixed=fixed, online=live, decode_speedup=live["tokens_per_s"] / fixed["tokens_per_s"])
    log(f"controller: fixed split {fixed['tokens_per_s']:.2f} tokens/s, online {live['tokens_per_s']:.2f} "
        f"({res['decode_speedup']:.3f}x); moves " + ", ".join(f"step {m['step']}: cap {m['cap']}" for m in live["moves"])
        + "; per regime " + ", ".join(f"{k} {v['tokens_per_s']:.1f} vs {fixed['per_regime'][k]['tokens_per_s']:.1f} "
                                       f"(over pool {v['steps_over_pool']} vs {fixed['per_regime'][k]['steps_over_pool']})"
                                       for k, v in live["per_regime"].items()))
    return res


PREFETCH_CAPS = (8, 16, 32)
PREFETCH_HORIZON = 4
PREFETCH_GAMMA = 0.5
PREFETCH_HINT_PRECISIONS = (1.0, 0.5, 0.25)


def prefetch_leg(run, wl, wisp, torch, warmup=16, steps=96):
    """Speculative prefetch (Sec. 4) on the decode workload, host pager, per-layer caps 8/16/32: no
    prefetch; the online co-activation predictor of App. E (fresh each arm, top-k of each layer
    prefetched before it is routed, source layers within PREFETCH_HORIZON, decay PREFETCH_GAMMA); and
    hints of a controlled precision (each step's true routing with a fraction 1 - p of the ids replaced
    by experts the step does not use, p in PREFETCH_HINT_PRECISIONS; p = 1 is a perfect predictor).
    The synthetic hidden states carry no cross-layer signal, so the co-activation predictor is near
    chance here; the hint arms stand in for predictors of the paper's quality (about 0.5 next-expert
    precision, App. E).  Tokens/s, demand faults and prefetch copies per token, and the measured
    precision (copies the step then used / copies issued)."""
    import numpy as np

    from paper_2606_21868_amd.workloads import degraded_hints
    steps = min(steps, run.steps - warmup)
    out = []
    run.ctx.set_pager(wisp.PAGER_HOST)
    for cap in PREFETCH_CAPS:
        if cap > wl.N:
            continue
        assert run.set_cap(cap) == cap
        arms = {}
        trace = None
        for arm in ("off", "predictor") + tuple(f"hints_p{p:g}" for p in PREFETCH_HINT_PRECISIONS):
            run.ctx.masters_ready()
            pred = None
            hints = None
            if arm == "predictor":
                pred = wisp.Predictor(wl.L, wl.N, PREFETCH_HORIZON, PREFETCH_GAMMA)
                run.ctx.set_prefetch(wisp.PREFETCH_PREDICTOR, pred, wl.k)
            elif arm.startswith("hints"):
                run.ctx.set_prefetch(wisp.PREFETCH_HINTS)
                hints = degraded_hints(trace, wl.N, float(arm[len("hints_p"):]), seed=cap)
            run.decode(record=False, steps=warmup, start=0, hints=hints[:warmup] if hints is not None else None)
            run.ctx.reset_stats()
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            o = run.decode(record=arm == "off", steps=steps, start=warmup,
                           hints=hints[warmup:] if hints is not None else None)
            torch.cuda.synchronize()
            el = time.perf_counter() - t0
            st = run.ctx.prefetch_stats()
            run.ctx.set_prefetch(wisp.PREFETCH_OFF)
            if pred is not None:
                pred.close()
            if arm == "off":
                full = run.decode(record=True, steps=warmup, start=0)   # the warmup steps' routing
                trace = np.concatenate([full["idx"], o["idx"]])
            n_tok = wl.T * steps
            arms[arm] = dict(tokens_per_s=n_tok / el, demand_faults_per_token=float(o["misses"].sum()) / n_tok,
                             prefetch_copies_per_token=st["issued"] / n_tok,
                             precision=st["useful"] / st["issued"] if st["issued"] else None,
                             link_GB_per_token=(float(o["misses"].sum()) + st["issued"]) * wl.blob / n_tok / 1e9)
            if hints is not None:
                arms[arm]["hint_precision"] = float(arm[len("hints_p"):])
        base = arms["off"]["tokens_per_s"]
        row = dict(cap=cap, **{a: v for a, v in arms.items()},
                   speedup={a: v["tokens_per_s"] / base for a, v in arms.items() if a != "off"})
        out.append(row)
        log(f"prefetch C={cap:3d}: off {base:6.2f} tokens/s; " + "; ".join(
            f"{a} {v['tokens_per_s']:6.2f} ({v['tokens_per_s'] / base:.2f}x, precision {v['precision'] or 0:.2f}, "
            f"{v['prefetch_copies_per_token']:.1f} copies + {v['demand_faults_per_token']:.1f} faults per token)"
            for a, v in arms.items() if a != "off"))
    assert run.set_cap(wl.cap) == wl.cap
    return out


# bounded decode legs of the workloads whose masters exceed the pinned memory of the test machines:
# (workload, warmup steps, timed steps), each from cold slot tables
PAGEABLE_LEGS = (("mixtral-8x7b-decode", 2, 6), ("deepseek-v3-16l-decode", 8, 64))


def pageable_leg(wisp, torch, name, warmup, steps, cpu=True):
    """Paged decode of a workload with pageable masters (every fault staged through the pinned bounce
    ring, host pager): tokens/s over `steps` timed steps after `warmup` steps from cold tables; the
    path roofline with the link term at the measured rate of that staged path; the expert gate/up
    kernel's HBM rate in the timed region; and the CPU oracle on a bounded sample."""
    from paper_2606_21868_amd.workloads import WORKLOADS
    wl = WORKLOADS[name]
    run = wisp.DecodeRun(wl, device=0, steps=warmup + steps, pageable=True)
    try:
        t0 = time.time()
        run.generate()
        gen_s = time.time() - t0
        n_probe = max(1, math.ceil(2e9 / wl.blob))
        link = run.ctx.probe_h2d(n_probe, 3)
        assert run.set_cap(wl.cap) == wl.cap
        run.ctx.masters_ready()
        run.decode(record=False, steps=warmup, start=0)
        run.ctx.reset_stats()
        run.ctx.reset_kernel_times()
        run.ctx.set_profiling(1 << wisp.K_FFN_GATEUP)
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        out = run.decode(record=False, steps=steps, start=warmup)
        torch.cuda.synchronize()
        el = time.perf_counter() - t1
        run.ctx.set_profiling(0)
        g = run.ctx.kernel_times(wisp.K_FFN_GATEUP)
        hits, misses = out["hits"], out["misses"]
        n_tok = wl.T * steps
        hbm_bytes = (float((hits + misses).sum()) + (wl.L * steps if wl.has_shared else 0)) * wl.blob + \
            wl.N * wl.d * 4 * wl.L * steps
        link_bytes = float(misses.sum()) * wl.blob
        t_roof = hbm_bytes / (HBM_PEAK_GBPS * 1e9) + link_bytes / (link * 1e9)
        gate = None
        if g["launches"]:
            gbps = g["bytes"] / (g["total_ms"] * 1e-3) / 1e9
            tr = measured_traffic(wl.name, "ffn_gateup")
            gate = dict(bound="hbm", kernel="ffn_rows expert gate/up (W1+W3 rows" +
                        (", fp8 E4M3 x bf16 block scales" if wl.w_dtype == wisp.FP8 else ", bf16") + "), timed region",
                        achieved=gbps, peak=HBM_PEAK_GBPS, unit="GB/s", frac=gbps / HBM_PEAK_GBPS,
                        launches=g["launches"], avg_launch_us=g["total_ms"] * 1e3 / g["launches"],
                        bytes_per_launch=g["bytes"] / g["launches"], traffic=tr["bytes_per_launch"] if tr else None,
                        traffic_detail=tr)
        res = dict(workload=wl.description, tokens_per_s=n_tok / el, ms_per_step=el / steps * 1e3, steps=steps,
                   warmup=warmup, cap_per_layer=wl.cap, generate_s=gen_s, masters="pageable (staged through a "
                   "pinned bounce ring)",
                   path_roofline=dict(t_roof_s=t_roof, t_measured_s=el, frac=t_roof / el,
                                      roofline_tokens_per_s=n_tok / t_roof, link_engine="copy_engine_staged",
                                      link_GBps_measured=link, hbm_peak_GBps=HBM_PEAK_GBPS,
                                      hbm_bytes_per_token=hbm_bytes / n_tok, link_bytes_per_token=link_bytes / n_tok,
                                      faults_per_token=float(misses.sum()) / n_tok),
                   gateup_kernel=gate)
        log(f"{name}: {steps} steps in {el:.2f} s -> {n_tok / el:.3f} tokens/s, {t_roof / el:.3f} of the path "
            f"roofline (staged link {link:.1f} GB/s, {float(misses.sum()) / n_tok:.1f} faults per token)"
            + (f"; gate/up {gate['achieved']:.0f} GB/s ({gate['frac']:.3f} of HBM)" if gate else ""))
        if cpu:
            res["cpu_baseline"] = cpu_baseline(run, wl, warmup, max_tokens=wl.T * 2, budget_s=10.0)
            log(f"{name}: cpu oracle {res['cpu_baseline']['value']:.4f} tokens/s ({res['cpu_baseline']['sample']})")
        return res
    finally:
        run.close()


def prefill_leg(wisp, torch, link, link_cu, passes=3):
    """Prefill tokens/s of the token-batch path (2048 tokens per layer, union 128 > C = 32, so four
    chunked Algorithm 1 steps per layer, grouped MFMA GEMMs), from cold slot tables each pass as the
    workload prescribes; then a fully resident pass (C = N, preloaded) for the matrix-core rate of
    the grouped GEMMs alone."""
    from paper_2606_21868_amd.workloads import WORKLOADS
    wl = WORKLOADS[PREFILL_WORKLOAD]
    run = wisp.DecodeRun(wl, device=0, steps=1)
    try:
        t0 = time.time()
        run.generate()
        log(f"prefill: generated {wl.L * wl.N} expert blobs and {wl.T} x {wl.L} token rows in {time.time() - t0:.1f} s")
        assert run.set_cap(wl.cap) == wl.cap
        times = []
        out = None
        for i in range(passes + 1):                    # the first pass is a warmup
            run.ctx.masters_ready()                    # cold: every slot empty
            torch.cuda.synchronize()
            t1 = time.perf_counter()
            out = run.decode(record=False, steps=1)
            torch.cuda.synchronize()
            if i > 0:
                times.append(time.perf_counter() - t1)
        times.sort()
        el = times[len(times) // 2]
        misses = int(out["misses"].sum())
        distinct = int((out["hits"] + out["misses"]).sum())
        pairs = wl.T * wl.k
        flops = 6.0 * wl.d * wl.I * pairs * wl.L
        # the token-batch fills stream by the compute units: the link term is the compute-unit rate; the
        # same roofline at the copy-engine rate is reported beside it
        t_link = misses * wl.blob / (link_cu * 1e9)
        t_hbm = distinct * wl.blob / (HBM_PEAK_GBPS * 1e9)
        t_mfma = flops / (MFMA_BF16_PEAK_TFLOPS * 1e12)
        t_roof = t_link + max(t_hbm, t_mfma)
        t_roof_ce = misses * wl.blob / (link * 1e9) + max(t_hbm, t_mfma)
        log(f"prefill: cold pass {el * 1e3:.1f} ms -> {wl.T / el:.0f} tokens/s, {t_roof / el:.3f} of the roofline "
            f"(compute-unit link rate; {t_roof_ce / el:.3f} at the copy-engine rate)")
        # fully resident: the same kernels with no faults; grouped GEMMs timed by HIP events
        assert run.set_cap(wl.N) == wl.N
        run.ctx.preload()
        run.decode(record=False, steps=1)
        mask = (1 << wisp.K_GROUPED_GATEUP) | (1 << wisp.K_GROUPED_DOWN) | (1 << wisp.K_PERMUTE) | \
               (1 << wisp.K_ROUTER_LOGITS) | (1 << wisp.K_ROUTER_SELECT) | (1 << wisp.K_COMBINE)
        rtimes = []
        for i in range(passes):
            if i == passes - 1:
                run.ctx.reset_kernel_times()
                run.ctx.set_profiling(mask)
            torch.cuda.synchronize()
            t1 = time.perf_counter()
            run.decode(record=False, steps=1)
            torch.cuda.synchronize()
            rtimes.append(time.perf_counter() - t1)
        run.ctx.set_profiling(0)
        kern = {}
        gflops, gbytes, gms = 0, 0, 0.0
        for kc in (wisp.K_GROUPED_GATEUP, wisp.K_GROUPED_DOWN, wisp.K_PERMUTE, wisp.K_ROUTER_LOGITS,
                   wisp.K_ROUTER_SELECT, wisp.K_COMBINE):
            t = run.ctx.kernel_times(kc)
            if not t["launches"]:
                continue
            e = dict(launches=t["launches"], avg_us=t["total_ms"] * 1e3 / t["launches"], total_ms=t["total_ms"])
            if t["bytes"]:
                e["GBps"] = t["bytes"] / (t["total_ms"] * 1e-3) / 1e9
            if t["flops"]:
                e["TFLOPs"] = t["flops"] / (t["total_ms"] * 1e-3) / 1e12
                gflops += t["flops"]
                gbytes += t["bytes"]
                gms += t["total_ms"]
            kern[wisp.KERNEL_CLASS_NAMES[kc]] = e
        achieved = gflops / (gms * 1e-3) / 1e12 if gms > 0 else None
        # what a plain streaming read of each GEMM launch's algorithmic bytes takes on this chip (fresh
        # windows of a buffer beyond the last-level cache): the practical floor of an HBM-bound launch
        floor = {}
        for kc in (wisp.K_GROUPED_GATEUP, wisp.K_GROUPED_DOWN):
            t = run.ctx.kernel_times(kc)
            if t["launches"] and t["bytes"]:
                nb = int(t["bytes"] // t["launches"]) // 16 * 16
                us = wisp.probe_hbm_read(nb, 20)
                name = wisp.KERNEL_CLASS_NAMES[kc]
                floor[name] = dict(bytes_per_launch=nb, us_per_launch=us, GBps=nb / (us * 1e-6) / 1e9,
                                   frac_of_peak=nb / (us * 1e-6) / 1e9 / HBM_PEAK_GBPS,
                                   kernel_frac_of_floor=us / kern[name]["avg_us"])
        if floor:
            log("prefill: plain read of the same bytes " + "; ".join(
                f"{k} {v['bytes_per_launch'] / 1e6:.0f} MB in {v['us_per_launch']:.1f} us = {v['GBps']:.0f} GB/s "
                f"(the GEMM at {v['kernel_frac_of_floor']:.2f} of it)" for k, v in floor.items()))
        mfma_peak = wisp.probe_mfma(10)   # the vendor's dense bf16 peak, checked on this chip
        log(f"prefill: matrix cores sustain {mfma_peak:.0f} TFLOP/s of dense bf16 on register operands "
            f"({mfma_peak / MFMA_BF16_PEAK_TFLOPS:.3f} of the 2.5 PFLOP/s peak)")
        rtimes.sort()
        rel = rtimes[len(rtimes) // 2]
        log(f"prefill: resident pass {rel * 1e3:.2f} ms -> {wl.T / rel:.0f} tokens/s; grouped GEMMs "
            f"{achieved:.0f} TFLOP/s ({achieved / MFMA_BF16_PEAK_TFLOPS:.3f} of the bf16 peak), "
            f"{gbytes / (gms * 1e-3) / 1e9:.0f} GB/s ({gbytes / (gms * 1e-3) / 1e9 / HBM_PEAK_GBPS:.3f} of HBM)")
        return dict(
            workload=wl.description, tokens_per_s=wl.T / el, pass_ms=el * 1e3, passes=len(times),
            pass_ms_all=[t * 1e3 for t in times], cap_per_layer=wl.cap, faults=misses, distinct_experts=distinct,
            roofline=dict(t_roof_s=t_roof, t_link_s=t_link, t_hbm_s=t_hbm, t_mfma_s=t_mfma, frac=t_roof / el,
                          roofline_tokens_per_s=wl.T / t_roof, link_engine="compute_units",
                          link_GBps_measured=link_cu, flops=flops,
                          side=dict(link_engine="copy_engine", link_GBps_measured=link, frac=t_roof_ce / el)),
            resident=dict(tokens_per_s=wl.T / rel, pass_ms=rel * 1e3, kernels=kern),
            mfma=dict(bound="mfma", achieved=achieved, peak=MFMA_BF16_PEAK_TFLOPS, unit="TFLOP/s",
                      frac=achieved / MFMA_BF16_PEAK_TFLOPS if achieved else None,
                      kernels="grouped gate/up + down (bf16 v_mfma_f32_32x32x16), resident pass",
                      peak_measured=mfma_peak, frac_of_measured_peak=achieved / mfma_peak if achieved else None,
                      peak_method="wisp_probe_mfma: register-only v_mfma_f32_32x32x16_bf16 stream, 8 waves per SIMD"),
            # at ~128 rows per expert the grouped GEMMs do ~100 FLOP per weight byte, below the bf16
            # ridge (2.5 PFLOP/s / 8 TB/s = 312): HBM is their bound
            hbm=dict(bound="hbm", achieved=gbytes / (gms * 1e-3) / 1e9 if gms > 0 else None, peak=HBM_PEAK_GBPS,
                     unit="GB/s", frac=gbytes / (gms * 1e-3) / 1e9 / HBM_PEAK_GBPS if gms > 0 else None,
                     kernels="grouped gate/up + down, algorithmic bytes (weights once, rows in and out)",
                     read_floor=floor,
                     frac_of_read_floor=(sum(v["us_per_launch"] * kern[k]["launches"] for k, v in floor.items()) /
                                         sum(kern[k]["total_ms"] * 1e3 for k in floor)) if floor else None))
    finally:
        run.close()


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None, help="timed decode steps (default: the run length minus warmup)")
    ap.add_argument("--warmup", type=int, default=16)
    ap.add_argument("--workload", default=None)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--kernel-timing", choices=["gateup", "all", "none"], default="gateup",
                    help="kernel classes bracketed by HIP events inside the timed region (default: the expert "
                         "gate/up GEMV, on which the roofline is reported)")
    ap.add_argument("--pager", choices=["both", "device", "host"], default="both",
                    help="which pager(s) to time; value is the device pager's when it runs")
    ap.add_argument("--no-prefill", action="store_true", help="skip the prefill leg")
    ap.add_argument("--no-sweep", action="store_true", help="skip the iso-VRAM budget sweep against static offload")
    ap.add_argument("--no-prefetch", action="store_true", help="skip the speculative-prefetch leg")
    ap.add_argument("--no-pageable", action="store_true",
                    help="skip the bounded Mixtral- and DeepSeek-shaped decode legs (pageable masters)")
    ap.add_argument("--no-fusion", action="store_true",
                    help="separate down and combine kernels instead of the fused down+combine (single-token steps)")
    ap.add_argument("--census-steps", type=int, default=24,
                    help="extra decode steps after the timed region with every kernel class timed (0 = skip)")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}, WORLD_SIZE {world}); the paged "
              f"MoE layer here runs per GPU and has no multi-GPU path.", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2606_21868_amd import wisp
    from paper_2606_21868_amd.workloads import BENCH_WORKLOAD, DTYPE_NAMES, WORKLOADS

    wl = WORKLOADS[args.workload or BENCH_WORKLOAD]
    if wl.prefill:
        raise SystemExit("prefill workloads are benchmarked by their own tests, not by this decode benchmark")
    warmup = max(0, args.warmup)
    steps = args.steps if args.steps is not None else wl.steps - warmup
    if steps < 1:
        raise SystemExit("need at least one timed step")
    total = warmup + steps
    log(f"workload {wl.name}: {warmup} warmup + {steps} timed steps, cap {wl.cap}")

    # master sets beyond the pinned memory a process may hold on the test machines are pageable (faults
    # staged through the bounce ring; host pager only)
    pageable_masters = wl.L * wl.N * wl.blob > PINNED_LIMIT_BYTES
    if pageable_masters:
        args.pager = "host"
    run = wisp.DecodeRun(wl, device=0, steps=total, pageable=pageable_masters)
    t0 = time.time()
    run.generate()
    log(f"generated {wl.L * wl.N} expert blobs ({wl.L * wl.N * wl.blob / 1e9:.1f} GB "
        f"{'pageable' if pageable_masters else 'pinned'}) and inputs in {time.time() - t0:.1f} s")
    n_probe = max(1, math.ceil(2e9 / wl.blob))
    link = run.ctx.probe_h2d(n_probe, 5)
    link_cu = run.ctx.probe_h2d(n_probe, 5, engine=wisp.LINK_CUS) if not pageable_masters else link
    hbm_copy = measure_hbm_copy(torch, wisp)
    log(f"host->device {link:.1f} GB/s copy engine, {link_cu:.1f} GB/s compute-unit streaming (median of 5 x "
        f"{n_probe} blobs); device copy {hbm_copy:.0f} GB/s")
    assert run.set_cap(wl.cap) == wl.cap
    run.ctx.set_fusion(not args.no_fusion)

    def timed_pass(pager, mask):
        """Cold slot tables, `warmup` untimed steps, then the timed steps; returns (elapsed, stats) of the
        timed steps and (elapsed, stats) of the warmup steps, which start from the cold tables."""
        run.ctx.masters_ready()                       # every slot empty: each pass starts cold
        run.ctx.set_pager(pager)
        warm = (0.0, None)
        if warmup:
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            w_out = run.decode(record=False, steps=warmup, start=0)
            torch.cuda.synchronize()
            warm = (time.perf_counter() - t0, w_out)
        run.ctx.reset_stats()
        run.ctx.reset_kernel_times()
        run.ctx.set_profiling(mask)
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        out = run.decode(record=False, steps=steps, start=warmup)
        torch.cuda.synchronize()
        el = time.perf_counter() - t1
        run.ctx.set_profiling(0)
        return el, out, warm

    def path_roofline(elapsed, out, n_steps=None, engine="copy_engine"):
        """T_roof with the link term at the measured rate of the engine that moves this pass's faults:
        the copy engine (hipMemcpyAsync, host pager) or the compute units (the device pager streams
        faulted experts with its own loads).  The other engine's rate is reported beside it."""
        n_steps = steps if n_steps is None else n_steps
        hits, misses = out["hits"], out["misses"]
        distinct = hits + misses
        hbm_bytes = float(distinct.sum()) * wl.blob + wl.N * wl.d * 4 * wl.L * n_steps
        link_bytes = float(misses.sum()) * wl.blob
        rate = {"copy_engine": link, "compute_units": link_cu}
        other = "compute_units" if engine == "copy_engine" else "copy_engine"
        t_roof = hbm_bytes / (HBM_PEAK_GBPS * 1e9) + link_bytes / (rate[engine] * 1e9)
        t_roof_other = hbm_bytes / (HBM_PEAK_GBPS * 1e9) + link_bytes / (rate[other] * 1e9)
        return dict(t_roof_s=t_roof, t_measured_s=elapsed, frac=t_roof / elapsed,
                    roofline_tokens_per_s=wl.T * n_steps / t_roof, link_engine=engine,
                    link_GBps_measured=rate[engine],
                    side=dict(link_engine=other, link_GBps_measured=rate[other], frac=t_roof_other / elapsed),
                    hbm_peak_GBps=HBM_PEAK_GBPS, device_copy_GBps_measured=hbm_copy,
                    hbm_bytes_per_token=hbm_bytes / (wl.T * n_steps), link_bytes_per_token=link_bytes / (wl.T * n_steps),
                    faults_per_token=float(misses.sum()) / (wl.T * n_steps),
                    fault_rate=float(misses.sum()) / float(distinct.sum()))

    def all_steps(el, out, warm, engine):
        """Every step of the pass from the cold tables (compulsory faults included): the warmup steps
        and the timed ones, each timed from its first route to its final device synchronisation."""
        w_el, w_out = warm
        if w_out is None:
            return None
        both = dict(hits=np.concatenate([w_out["hits"], out["hits"]]),
                    misses=np.concatenate([w_out["misses"], out["misses"]]))
        n = warmup + steps
        return dict(steps=n, tokens_per_s=wl.T * n / (w_el + el),
                    path_roofline=path_roofline(w_el + el, both, n, engine))

    def kernel_table():
        tab = {}
        for kc, name in enumerate(wisp.KERNEL_CLASS_NAMES):
            t = run.ctx.kernel_times(kc)
            if t["launches"]:
                tab[name] = dict(launches=t["launches"], avg_us=t["total_ms"] * 1e3 / t["launches"],
                                 total_ms=t["total_ms"],
                                 bytes_per_launch=t["bytes"] / t["launches"] if t["bytes"] else None,
                                 GBps=t["bytes"] / (t["total_ms"] * 1e-3) / 1e9 if t["bytes"] and t["total_ms"] > 0
                                 else None)
        return tab

    census_faults = {}

    def census(pager):
        # every class timed, on steps after the timed region (the events slow the path, so these
        # steps are not part of any throughput)
        if args.census_steps <= 0:
            return {}
        run.ctx.set_pager(pager)
        run.ctx.reset_kernel_times()
        run.ctx.set_profiling(True)
        o = run.decode(record=False, steps=min(args.census_steps, total), start=0)
        run.ctx.set_profiling(0)
        census_faults[pager] = o
        return kernel_table()

    def device_ffn_roofline(tab):
        # the device pager's gate/up kernel reads resident experts from HBM and streams faulted ones
        # over the host link: its floor is hit bytes / HBM peak + fault bytes / measured link, per launch
        o = census_faults.get(wisp.PAGER_DEVICE)
        g = tab.get("ffn_gateup")
        if o is None or not g:
            return None
        gate_bytes = 2 * wl.d * wl.I * (2 if wl.w_dtype == wisp.BF16 else 4)
        # the faulted experts stream by the kernel's own loads: the link term is the compute-unit rate
        t_roof = (float(o["hits"].sum()) * gate_bytes / (HBM_PEAK_GBPS * 1e9) +
                  float(o["misses"].sum()) * wl.blob / (link_cu * 1e9))
        t_meas = g["total_ms"] * 1e-3
        return dict(kernel="ffn_gateup_dev (resident experts from HBM, faulted ones streamed from pinned host memory)",
                    bound="hbm+link", launches=g["launches"], avg_launch_us=g["avg_us"], t_roof_s=t_roof,
                    t_measured_s=t_meas, frac=t_roof / t_meas, link_engine="compute_units",
                    link_GBps_measured=link_cu, hbm_peak_GBps=HBM_PEAK_GBPS,
                    source="census steps (every kernel class event-timed)")

    mask = {"gateup": 1 << wisp.K_FFN_GATEUP, "all": True, "none": 0}[args.kernel_timing]
    passes = {}
    roof = None
    if args.pager in ("both", "host"):
        el, out, warm = timed_pass(wisp.PAGER_HOST, mask)
        tk = kernel_table()
        passes["host"] = dict(tokens_per_s=wl.T * steps / el, ms_per_step=el / steps * 1e3,
                              path_roofline=path_roofline(el, out, engine="copy_engine"),
                              all_steps=all_steps(el, out, warm, "copy_engine"),
                              kernels_timed_region=tk, kernel_census=census(wisp.PAGER_HOST))
        log(f"host pager: {steps} steps in {el:.3f} s -> {wl.T * steps / el:.2f} tokens/s, "
            f"{passes['host']['path_roofline']['frac']:.3f} of the path roofline")
        if "ffn_gateup" in tk:
            g = tk["ffn_gateup"]
            tr = measured_traffic(wl.name, "ffn_gateup")
            roof = dict(bound="hbm", achieved=g["GBps"], peak=HBM_PEAK_GBPS, unit="GB/s", frac=g["GBps"] / HBM_PEAK_GBPS,
                        traffic=tr["bytes_per_launch"] if tr else None,
                        traffic_detail=tr, kernel=f"expert gate/up GEMV (W1+W3 rows, {DTYPE_NAMES[wl.w_dtype]} weights), "
                                                  f"host-pager pass",
                        avg_launch_us=g["avg_us"], bytes_per_launch=g["bytes_per_launch"], launches=g["launches"])
            # what a plain streaming read of the same bytes per launch takes on this GPU: the floor of
            # any kernel that must read them in one launch of this size
            nb = int(g["bytes_per_launch"]) // 16 * 16
            us = wisp.probe_hbm_read(nb, 400)
            floor = nb / (us * 1e-6) / 1e9
            roof["read_floor"] = dict(
                bytes_per_launch=nb, us_per_launch=us, GBps=floor, frac_of_peak=floor / HBM_PEAK_GBPS,
                method="plain streaming-read kernel, 400 launches back to back over windows of a 2 GiB buffer")
            roof["frac_of_read_floor"] = g["GBps"] / floor
            log(f"gate/up GEMV: {g['GBps']:.0f} GB/s in the timed region; a plain read of the same {nb / 1e6:.1f} MB per "
                f"launch: {us:.2f} us = {floor:.0f} GB/s ({g['GBps'] / floor:.3f} of it)")
    if args.pager in ("both", "device"):
        el, out, warm = timed_pass(wisp.PAGER_DEVICE, 0)
        passes["device"] = dict(tokens_per_s=wl.T * steps / el, ms_per_step=el / steps * 1e3,
                                path_roofline=path_roofline(el, out, engine="compute_units"),
                                all_steps=all_steps(el, out, warm, "compute_units"),
                                kernel_census=census(wisp.PAGER_DEVICE))
        passes["device"]["ffn_roofline"] = device_ffn_roofline(passes["device"]["kernel_census"])
        log(f"device pager: {steps} steps in {el:.3f} s -> {wl.T * steps / el:.2f} tokens/s, "
            f"{passes['device']['path_roofline']['frac']:.3f} of the path roofline")
    main_pass = "device" if "device" in passes else "host"
    tok_s = passes[main_pass]["tokens_per_s"]
    elapsed = steps / tok_s * wl.T
    path = passes[main_pass]["path_roofline"]

    sweep = None
    controller = None
    configurator = None
    if not args.no_sweep and wl.name == BENCH_WORKLOAD:
        sweep = sweep_leg(run, wl, wisp, torch)
        controller = controller_leg(run, wl, wisp, torch)
        configurator = configurator_leg(run, wl, wisp, torch, link_cu)
    prefetch = None
    if not args.no_prefetch and wl.name == BENCH_WORKLOAD:
        prefetch = prefetch_leg(run, wl, wisp, torch)
    cpu = None
    if not args.no_cpu_baseline:
        log("cpu baseline (oracle)")
        cpu = cpu_baseline(run, wl, warmup)
        log(f"cpu oracle {cpu['value']:.3f} tokens/s on {cpu['cores']} threads")
    run.close()
    prefill = None
    if not args.no_prefill:
        prefill = prefill_leg(wisp, torch, link, link_cu)
    pageable = None
    if not args.no_pageable and wl.name == BENCH_WORKLOAD:
        pageable = {name: pageable_leg(wisp, torch, name, w, n, cpu=not args.no_cpu_baseline)
                    for name, w, n in PAGEABLE_LEGS}

    result = {
        "metric": "paged MoE decode tokens/s at fixed VRAM expert budget",
        "value": tok_s,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": warmup,
        "ms_per_step": elapsed / steps * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": DTYPE_NAMES[wl.w_dtype],
        "data": "synthetic (seeded N(0,0.02) weights, AR(1) rho=0.9 hidden states)",
        "config": {"workload": wl.description, "layers": wl.L, "d_model": wl.d, "d_ff": wl.I, "experts": wl.N,
                   "top_k": wl.k, "batch": wl.T, "expert_budget_bytes": wl.budget_bytes, "cap_per_layer": wl.cap,
                   "expert_blob_bytes": wl.blob, "decode_steps": total},
        "roofline": roof,
        "path_roofline": path,
        "cpu_baseline": cpu,
        "pager": main_pass,
        "passes": passes,
        "kernel_timing": args.kernel_timing,
        "prefill": prefill,
        "sweep": sweep,
        "controller": controller,
        "configurator": configurator,
        "prefetch": prefetch,
        "pageable_legs": pageable,
    }
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
