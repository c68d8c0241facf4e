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
  controller     the live dual-resize (App. B): a fixed split's idle KV moved to expert slots by the
                 control law, decode tokens/s before and after;
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
MFMA_BF16_PEAK_TFLOPS = 2500.0      # dense bf16 matrix-core peak of the MI355X
PREFILL_WORKLOAD = "qwen3-30b-a3b-prefill"
TRAFFIC_SUMMARIES = {k: os.path.join(ROOT, "profiles", f"{k}_qwen3-30b-a3b-decode_hbm_traffic.txt")
                     for k in ("ffn_gateup",)}
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
    summary = TRAFFIC_SUMMARIES.get(kname)
    if workload != "qwen3-30b-a3b-decode" or summary is None or not os.path.exists(summary):
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
    """The oracle as it stands: fully resident fp64 layer, all layers of consecutive decode steps."""
    import oracle
    threads = oracle.num_threads()
    t0 = time.perf_counter()
    tokens = 0
    s = start_step
    while tokens < max_tokens and s < run.x_host.shape[1]:
        for l in range(wl.L):
            oracle.moe_layer(wl.route, run.master_ptrs(l), run.wr_host[l], run.x_host[l, s], wl.k, wl.I, wl.w_dtype,
                             run.shared_ptr(l), wl.n_groups, wl.topk_groups)
        tokens += wl.T
        s += 1
        if time.perf_counter() - t0 > budget_s:
            break
    dt = time.perf_counter() - t0
    return dict(value=tokens / dt, unit="tokens/s", cores=threads, kind="oracle",
                sample=f"{tokens // wl.T} decode step(s) x {wl.L} layers x batch {wl.T} "
                       f"(fully resident fp64 layer, weights read from the same pinned host masters), {dt:.1f} s")


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
        paged = timed(lambda n: run.decode(record=False, steps=n, start=warmup, stats=False), steps)
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
                        zero_copy_offload_tokens_per_s=zc[0], zero_copy_resident_layers=zc[1],
                        speedup_vs_zero_copy=paged / zc[0],
                        bulk_offload_tokens_per_s=st[0], bulk_resident_layers=st[1],
                        speedup_vs_bulk=paged / st[0]))
        log(f"sweep C={cap:3d} ({budget / 1e9:5.1f} GB): paged {paged:7.2f} tokens/s; zero-copy offload {zc[0]:7.2f} "
            f"({zc[1]} resident layers) -> {paged / zc[0]:4.1f}x; bulk offload {st[0]:7.2f} ({st[1]}) -> "
            f"{paged / st[0]:5.1f}x")
    return out


# Qwen3-30B-A3B KV cache: 48 layers x (K, V) x 4 KV heads x 128 x bf16 per token, 16-token blocks
KV_BLOCK_BYTES = 16 * 48 * 2 * 4 * 128 * 2
KV_POOL_GIB = 2.79          # the fixed split's KV pool in the paper's live run
KV_PEAK_FRACTION = 0.44     # its observed peak occupancy
KV_HEADROOM = 0.2


def controller_leg(run, wl, wisp, torch, warmup=16, steps=96):
    """The live dual-resize of Sec. 3.5 / App. B on the decode workload: a fixed split (cap 32 and a
    2.79 GiB KV pool of real device memory) serves a burst whose KV peaks at 44 % of the pool; at the
    drained barrier the control law (Eqs. 6-8) moves the idle KV to expert slots and the move is
    applied (KV shrunk first, then the scratch grown).  Decode tokens/s are timed before and after on
    the same steps (the KV cache itself is simulated: its bytes are held, not read)."""
    steps = min(steps, run.steps - warmup)
    a = wl.L * wl.blob
    b = KV_BLOCK_BYTES
    kv0 = int(KV_POOL_GIB * (1 << 30)) // b
    B = wl.cap * a + kv0 * b

    def measure():
        run.ctx.set_pager(wisp.PAGER_HOST)
        run.ctx.masters_ready()
        run.ctx.set_pager(wisp.PAGER_DEVICE)
        run.decode(record=False, steps=warmup, start=0, stats=False)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        run.decode(record=False, steps=steps, start=warmup, stats=False)
        torch.cuda.synchronize()
        return wl.T * steps / (time.perf_counter() - t0)

    run.ctx.set_pager(wisp.PAGER_HOST)
    assert run.set_cap(wl.cap) == wl.cap
    pool = wisp.KvPool(b, kv0)
    try:
        fixed = measure()
        run.ctx.set_pager(wisp.PAGER_HOST)
        cap, kv, move = wisp.resize_target(B, a, b, 0, KV_HEADROOM, 1, wl.N, 1, int(KV_PEAK_FRACTION * kv0), wl.cap)
        t0 = time.perf_counter()
        if move:
            wisp.dual_resize(run.ctx, pool, cap, kv)
        move_s = time.perf_counter() - t0
        dyn = measure()
        res = dict(budget_GiB=B / (1 << 30), kv_block_bytes=b,
                   fixed=dict(cap=wl.cap, kv_GiB=kv0 * b / (1 << 30), tokens_per_s=fixed),
                   dynamic=dict(cap=run.ctx.cap(), kv_GiB=pool.blocks * b / (1 << 30), tokens_per_s=dyn),
                   move_seconds=move_s, decode_speedup=dyn / fixed)
        log(f"controller: cap {wl.cap} / KV {kv0 * b / (1 << 30):.2f} GiB -> cap {run.ctx.cap()} / KV "
            f"{pool.blocks * b / (1 << 30):.2f} GiB (move {move_s * 1e3:.0f} ms); decode {fixed:.2f} -> {dyn:.2f} "
            f"tokens/s ({dyn / fixed:.3f}x)")
        return res
    finally:
        pool.close()


PREFETCH_CAPS = (8, 16, 32)
PREFETCH_HORIZON = 4
PREFETCH_GAMMA = 0.5


def prefetch_leg(run, wl, wisp, torch, warmup=16, steps=96):
    """Speculative prefetch (Sec. 4) on the decode workload, host pager, per-layer caps 8/16/32: no
    prefetch; the online co-activation predictor of App. E (fresh each arm, top-k of each layer
    prefetched before it is routed, source layers within PREFETCH_HORIZON, decay PREFETCH_GAMMA); and
    perfect hints (each step's true routing).  Tokens/s, demand faults and prefetch copies per
    token, and the predictor's precision (prefetched experts the next step used / copies)."""
    import numpy as np
    steps = min(steps, run.steps - warmup)
    out = []
    run.ctx.set_pager(wisp.PAGER_HOST)
    for cap in PREFETCH_CAPS:
        if cap > wl.N:
            continue
        assert run.set_cap(cap) == cap
        arms = {}
        trace = None
        for arm in ("off", "predictor", "perfect"):
            run.ctx.masters_ready()
            pred = None
            if arm == "predictor":
                pred = wisp.Predictor(wl.L, wl.N, PREFETCH_HORIZON, PREFETCH_GAMMA)
                run.ctx.set_prefetch(wisp.PREFETCH_PREDICTOR, pred, wl.k)
            elif arm == "perfect":
                run.ctx.set_prefetch(wisp.PREFETCH_HINTS)
            hints = trace.reshape(trace.shape[0], wl.L, -1) if arm == "perfect" else None
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
        row = dict(cap=cap, **{a: v for a, v in arms.items()},
                   predictor_speedup=arms["predictor"]["tokens_per_s"] / arms["off"]["tokens_per_s"],
                   perfect_speedup=arms["perfect"]["tokens_per_s"] / arms["off"]["tokens_per_s"])
        out.append(row)
        pr = arms["predictor"]
        log(f"prefetch C={cap:3d}: off {arms['off']['tokens_per_s']:6.2f} tokens/s; predictor {pr['tokens_per_s']:6.2f} "
            f"({row['predictor_speedup']:.2f}x, precision {pr['precision'] or 0:.2f}, "
            f"{pr['prefetch_copies_per_token']:.1f} copies + {pr['demand_faults_per_token']:.1f} faults per token); "
            f"perfect hints {arms['perfect']['tokens_per_s']:6.2f} ({row['perfect_speedup']:.2f}x)")
    assert run.set_cap(wl.cap) == wl.cap
    return out


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
                     kernels="grouped gate/up + down, algorithmic bytes (weights once, rows in and out)"))
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

    run = wisp.DecodeRun(wl, device=0, steps=total)
    t0 = time.time()
    run.generate()
    log(f"generated {wl.L * wl.N} expert blobs ({wl.L * wl.N * wl.blob / 1e9:.1f} GB pinned) and inputs in "
        f"{time.time() - t0:.1f} s")
    n_probe = max(1, math.ceil(2e9 / wl.blob))
    link = run.ctx.probe_h2d(n_probe, 5)
    link_cu = run.ctx.probe_h2d(n_probe, 5, engine=wisp.LINK_CUS)
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
                        traffic_detail=tr, kernel="ffn_rows<bf16,bf16,gate/up> expert GEMV (W1+W3 rows), host-pager pass",
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
    if not args.no_sweep and wl.name == BENCH_WORKLOAD:
        sweep = sweep_leg(run, wl, wisp, torch)
        controller = controller_leg(run, wl, wisp, torch)
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
        "prefetch": prefetch,
    }
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
