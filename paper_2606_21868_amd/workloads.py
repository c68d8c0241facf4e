"""Workload shapes of the paged MoE layer (synthetic stand-ins for the paper's models).

Each workload fixes the layer shape, the routing variant, the weight format, the run length and
the VRAM expert budget.  The per-layer cap follows C = floor(B_exp / (L * M_e)) (WiSP Sec. 3.1),
with B_exp in decimal bytes.  Weights ~ N(0, 0.02^2); router W_r ~ N(0, 1/d) in fp32; decode
hidden states are AR(1) chains (rho 0.9) per (layer, batch row); prefill states are i.i.d. N(0, I).
"""
from __future__ import annotations

from dataclasses import dataclass, replace

F32, BF16, FP8 = 0, 1, 2
ROUTE_SOFTMAX_RENORM, ROUTE_TOPK_SOFTMAX, ROUTE_SIGMOID_GROUP = 0, 1, 2
DTYPE_NAMES = {F32: "f32", BF16: "bf16", FP8: "fp8e4m3-b128"}


def blob_bytes(w_dtype: int, d: int, I: int) -> int:
    """Bytes of one expert blob: W1 | W3 | W2 (+ bf16 128x128 block scales for fp8)."""
    n = d * I
    if w_dtype == F32:
        return 12 * n
    if w_dtype == BF16:
        return 6 * n
    return 3 * n + 2 * 3 * (d // 128) * (I // 128)


@dataclass(frozen=True)
class Workload:
    name: str
    description: str
    L: int            # MoE layers
    d: int            # model width
    I: int            # expert intermediate width
    N: int            # routed experts per layer
    k: int            # experts per token
    T: int            # tokens per step (batch rows in decode; prompt tokens in prefill)
    steps: int        # decode steps (1 for a prefill pass)
    w_dtype: int
    x_dtype: int
    route: int
    budget_bytes: int  # VRAM expert budget B_exp (decimal bytes)
    n_groups: int = 1
    topk_groups: int = 1
    has_shared: bool = False
    prefill: bool = False
    seed: int = 0

    @property
    def blob(self) -> int:
        return blob_bytes(self.w_dtype, self.d, self.I)

    @property
    def cap(self) -> int:
        return self.budget_bytes // (self.L * self.blob)

    def with_(self, **kw) -> "Workload":
        return replace(self, **kw)


def _budget_slots(slots_total: int, w_dtype: int, d: int, I: int) -> int:
    return slots_total * blob_bytes(w_dtype, d, I)


WORKLOADS = {
    "tiny-fp32": Workload(
        "tiny-fp32", "1-layer tiny MoE, d=256, 8 experts top-2 (softmax then renormalise), I=512, fp32, "
        "batch 1, 64 decode steps, 4 expert slots",
        L=1, d=256, I=512, N=8, k=2, T=1, steps=64, w_dtype=F32, x_dtype=F32, route=ROUTE_SOFTMAX_RENORM,
        budget_bytes=_budget_slots(4, F32, 256, 512)),
    "qwen3-30b-a3b-decode": Workload(
        "qwen3-30b-a3b-decode", "Qwen3-30B-A3B-shaped paged decode: 48 layers, d=2048, 128 experts top-8 "
        "(softmax then renormalise), I=768, bf16, batch 1, 512 steps, budget 25% of 6144 experts (C=32)",
        L=48, d=2048, I=768, N=128, k=8, T=1, steps=512, w_dtype=BF16, x_dtype=BF16,
        route=ROUTE_SOFTMAX_RENORM, budget_bytes=_budget_slots(1536, BF16, 2048, 768)),
    "qwen3-30b-a3b-prefill": Workload(
        "qwen3-30b-a3b-prefill", "Qwen3-30B-A3B-shaped prefill chunk: same weights and routing, 2048 i.i.d. "
        "tokens, one pass, budget 25% (C=32)",
        L=48, d=2048, I=768, N=128, k=8, T=2048, steps=1, w_dtype=BF16, x_dtype=BF16,
        route=ROUTE_SOFTMAX_RENORM, budget_bytes=_budget_slots(1536, BF16, 2048, 768), prefill=True),
    "mixtral-8x7b-decode": Workload(
        "mixtral-8x7b-decode", "Mixtral-8x7B-shaped paged decode: 32 layers, d=4096, 8 experts top-2 "
        "(softmax over the top-2 logits), I=14336, bf16, batch 4, 256 steps, 64 of 256 slots (C=2)",
        L=32, d=4096, I=14336, N=8, k=2, T=4, steps=256, w_dtype=BF16, x_dtype=BF16,
        route=ROUTE_TOPK_SOFTMAX, budget_bytes=_budget_slots(64, BF16, 4096, 14336)),
    "deepseek-v3-16l-decode": Workload(
        "deepseek-v3-16l-decode", "DeepSeek-V3-shaped paged decode, 16 layers: d=7168, 256 routed + 1 "
        "shared expert, I=2048, sigmoid routing limited to 4 of 8 groups then top-8 renormalised, fp8 E4M3 "
        "with bf16 128x128 block scales, batch 1, 256 steps, 40 GB expert budget (C=56)",
        L=16, d=7168, I=2048, N=256, k=8, T=1, steps=256, w_dtype=FP8, x_dtype=BF16,
        route=ROUTE_SIGMOID_GROUP, budget_bytes=40_000_000_000, n_groups=8, topk_groups=4, has_shared=True),
}

def degraded_hints(idx, n_experts, precision, seed=0):
    """Prefetch hints of a chosen precision for the speculative-prefetch experiment (Sec. 4): for each
    (step, layer) of a routing trace idx [S, L, T, k], the distinct routed ids with a fraction
    1 - precision of them (rounded) replaced by ids drawn without replacement from the experts that
    step does not route to, in a seeded random order.  Returns hints [S, L, n] int32, n the largest
    routed-set size, padded with -1.  precision 1 gives the true routing (a perfect predictor)."""
    import numpy as np
    rng = np.random.default_rng(seed)
    S, L = idx.shape[:2]
    sets = [[np.unique(idx[s, l]) for l in range(L)] for s in range(S)]
    n = max(len(r) for row in sets for r in row)
    out = np.full((S, L, n), -1, np.int32)
    for s in range(S):
        for l in range(L):
            r = sets[s][l]
            m = int(round(len(r) * (1.0 - precision)))
            others = np.setdiff1d(np.arange(n_experts), r)
            m = min(m, others.size)
            keep = rng.choice(r, size=len(r) - m, replace=False)
            wrong = rng.choice(others, size=m, replace=False)
            h = rng.permutation(np.concatenate([keep, wrong]))
            out[s, l, :h.size] = h
    return out


KV_REGIMES = {
    # per-session context at the start of a turn, as a fraction of a session's share of the initial KV
    # pool, and the chance per decode step that a session's turn ends (a new one starts)
    "tool": (0.15, 0.55, 0.08),      # short tool-call bursts: the pool is mostly idle
    "long": (0.75, 1.00, 0.01),      # long-context turns: the pool is nearly full
}


def kv_occupancy_trace(regimes, pool_blocks, sessions=4, block_tokens=16, seed=0):
    """A seeded KV-occupancy trace (blocks in use after each decode step) for the online allocator of
    Sec. 3.5: `sessions` concurrent sessions whose contexts grow by one token per step; a turn ends with
    the regime's probability and the next starts at a context drawn from the regime's range.  Every
    session starts a new turn when the regime changes.  regimes: [(steps, "tool" | "long")].  Returns
    int64 [sum of steps]."""
    import numpy as np
    rng = np.random.default_rng(seed)
    share = pool_blocks / sessions
    out = []
    for steps, kind in regimes:
        lo, hi, p_end = KV_REGIMES[kind]
        ctx = rng.uniform(lo, hi, sessions) * share * block_tokens          # tokens
        for _ in range(steps):
            ends = rng.random(sessions) < p_end
            ctx[ends] = rng.uniform(lo, hi, int(ends.sum())) * share * block_tokens
            ctx += 1.0
            out.append(int(np.ceil(ctx / block_tokens).sum()))
    return np.array(out, np.int64)


# The benchmarked workload: the paged decode on which the decode-throughput metric is quoted.
BENCH_WORKLOAD = "qwen3-30b-a3b-decode"
