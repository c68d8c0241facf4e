"""GPU tests of the staged fill path: expert masters in pageable host memory, faults copied through
the pinned bounce ring.

After every decode step, each slot whose occupant changed in that step is read back and compared
byte for byte with its master (so a piece that landed wrong is named by layer, slot, expert and
offset), and the step's outputs are checked against the oracle.  A wrong output with intact slots
points at the ordering between the fills and the kernels that read them; a wrong slot points at the
staging itself.  The Qwen3 case faults one 9.4 MB blob (one staging piece) at a time; the
Mixtral-width case faults 352 MB blobs (eleven pieces) in chunked Algorithm 1 steps at batch 4.
"""
import numpy as np
import pytest

from parity import check_run, log
from paper_2606_21868_amd import wisp
from paper_2606_21868_amd.workloads import WORKLOADS

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu


def _first_difference(a, b):
    ne = np.flatnonzero(a != b)
    return (int(ne[0]), int(ne[-1]), int(ne.size)) if ne.size else None


@pytest.mark.parametrize("name,shape,cap,steps", [
    ("qwen3-30b-a3b-decode", dict(L=4), 32, 48),
    ("mixtral-8x7b-decode", dict(L=1, T=4), 2, 12),
])
def test_staged_fills_land_intact_every_step(name, shape, cap, steps):
    wl = WORKLOADS[name].with_(**shape)
    log(f"[case] staged fills {wl.name} {shape} C={cap} steps={steps}")
    run = wisp.DecodeRun(wl, device=0, steps=steps, pageable=True)
    try:
        run.generate()
        assert run.set_cap(cap) == cap
        masters = {}
        y = np.zeros((steps, wl.L, wl.T, wl.d), np.float32)
        idx = np.zeros((steps, wl.L, wl.T, wl.k), np.int32)
        w = np.zeros((steps, wl.L, wl.T, wl.k), np.float32)
        occ = [[-1] * cap for _ in range(wl.L)]
        filled = 0
        for s in range(steps):
            out = run.decode(record=True, steps=1, start=s)
            y[s], idx[s], w[s] = out["y"][0], out["idx"][0], out["w"][0]
            for l in range(wl.L):
                for slot in range(cap):
                    e = run.ctx.expert_in_slot(l, slot)
                    if e < 0 or e == occ[l][slot]:
                        continue
                    occ[l][slot] = e
                    if (l, e) not in masters:
                        masters[(l, e)] = run.master_blob(l, e)
                    diff = _first_difference(run.ctx.read_slot(l, slot, run.blob_bytes), masters[(l, e)])
                    assert diff is None, (f"step {s} layer {l} slot {slot} expert {e}: bytes {diff[0]}..{diff[1]} "
                                          f"differ ({diff[2]} bytes) from the master")
                    filled += 1
        pts = [(s, l) for s in range(steps) for l in range(wl.L)]
        _, _, _, worst, _ = check_run(run, dict(idx=idx, w=w, y=y), steps, pts)
        log(f"  {filled} filled slots byte-equal to their masters; outputs within tolerance (worst {worst:.2e})")
    finally:
        run.close()
