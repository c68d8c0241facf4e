"""CPU checks of the workload helpers: the controlled-precision prefetch hints."""
import numpy as np
import pytest

from paper_2606_21868_amd.workloads import degraded_hints


@pytest.mark.parametrize("p", [1.0, 0.5, 0.25, 0.0])
def test_degraded_hints_have_the_asked_precision(p):
    rng = np.random.default_rng(1)
    idx = np.stack([[rng.permutation(128)[:8] for _ in range(3)] for _ in range(5)])[:, :, None, :]
    h = degraded_hints(idx, 128, p, seed=3)
    assert h.shape == (5, 3, 8)
    for s in range(5):
        for l in range(3):
            hs = set(h[s, l].tolist())
            assert -1 not in hs and len(hs) == 8 and max(hs) < 128
            assert len(hs & set(idx[s, l, 0].tolist())) == round(8 * p)
    assert np.array_equal(h, degraded_hints(idx, 128, p, seed=3))


def test_degraded_hints_of_batched_steps_use_the_union():
    idx = np.array([[[[0, 1], [1, 2]]]])           # one step, one layer, two tokens: union {0, 1, 2}
    h = degraded_hints(idx, 8, 1.0)
    assert sorted(h[0, 0].tolist()) == [0, 1, 2]
