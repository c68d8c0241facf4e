"""GPU parity of the Mixtral-8x7B-shaped decode workload at full size, over all of its 256 steps
(32 layers x 8 experts of 352 MB, 90.2 GB of masters, batch 4, C = 2).  Unions of up to 8 experts per
layer-step against 2 slots make every step several chunked Algorithm 1 steps, and each step moves
about 42 GB over the host link, so the run takes minutes.  The masters exceed the pinned memory a
process may hold on the test machines (65 GiB): they are pageable and every fault is staged
through the pinned bounce ring.

The run is split into tests of 32 steps each that share one context (module fixture) and continue
its slot tables; any of them run alone first decodes the steps before its own.  The last test checks
every routing decision, gate and paging count of the 256 steps against the oracle, outputs at sampled
(step, layer) points and every exempt token, the masters, and bit identity with the fully resident run.
Collected after the other GPU tests (longest).
"""
import numpy as np
import pytest

from parity import check_masters_unchanged, check_run, log
from paper_2606_21868_amd.workloads import WORKLOADS

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

WL = WORKLOADS["mixtral-8x7b-decode"]
CHUNK = 32
N_CHUNKS = WL.steps // CHUNK


class _State:
    def __init__(self):
        from paper_2606_21868_amd import wisp
        log(f"[case] {WL.name} full size L={WL.L} d={WL.d} I={WL.I} N={WL.N} k={WL.k} T={WL.T} "
            f"steps={WL.steps} C={WL.cap} (pageable masters)")
        self.run = wisp.DecodeRun(WL, device=0, steps=WL.steps, pageable=True)
        self.run.generate()
        log(f"  generated in {self.run.gen_seconds:.1f}s")
        assert self.run.set_cap(WL.cap) == WL.cap
        self.done = 0
        self.parts = []

    def advance(self, upto):
        while self.done < upto:
            o = self.run.decode(record=True, steps=CHUNK, start=self.done)
            self.parts.append(o)
            self.done += CHUNK
            log(f"  steps {self.done - CHUNK}..{self.done - 1}: {int(o['misses'].sum())} faults, "
                f"{int(o['chunks'].max())} chunks at most per layer-step")

    def joined(self):
        return {k: np.concatenate([p[k] for p in self.parts]) for k in ("idx", "w", "y", "hits", "misses", "chunks")}


@pytest.fixture(scope="module")
def state():
    st = _State()
    yield st
    st.run.close()


@pytest.mark.parametrize("chunk", range(N_CHUNKS))
def test_mixtral_full_size_steps(state, chunk):
    state.advance((chunk + 1) * CHUNK)
    assert state.parts[chunk]["chunks"].max() > 1


def test_mixtral_full_size_parity(state):
    state.advance(WL.steps)
    run, out = state.run, state.joined()
    steps = WL.steps
    pts = [(0, 0), (3, 9), (40, 31), (97, 16), (150, 4), (201, 22), (steps - 1, WL.L - 1)]
    used = sorted({(l, int(e)) for s, l in pts for e in np.unique(out["idx"][s, l])})
    assert not check_masters_unchanged(run, used[:16])
    _, exempt, reordered, worst, _ = check_run(run, out, steps, pts, cap=WL.cap)
    log(f"  routing, gates and paging of all {steps} steps match the oracle ({len(exempt)} near-tie tokens "
        f"exempt, {len(reordered)} reordered); outputs at {len(pts)} points, worst row-relative error {worst:.2e}; "
        f"{int(out['misses'].sum())} faults")
    # fully resident: C = N, preloaded, same kernels -> bit-identical over every step, no faults
    assert run.set_cap(WL.N) == WL.N
    run.ctx.preload()
    run.ctx.reset_stats()
    res = run.decode(record=True, steps=steps, start=0)
    assert int(res["misses"].sum()) == 0
    assert np.array_equal(res["idx"], out["idx"])
    assert np.array_equal(res["y"].view(np.uint32), out["y"].view(np.uint32)), "paged != resident bits"
    log(f"  paged output bit-identical to the fully resident run over all {steps} steps")
