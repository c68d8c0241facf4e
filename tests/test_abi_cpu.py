"""Host-only checks of the C-ABI library: it loads, exports every declared symbol, validates
descriptions before touching the GPU, and its slot table (the pager's host logic) agrees with the
oracle's independent Algorithm 1 simulator."""
import os
import re

import numpy as np
import pytest

import oracle
from paper_2606_21868_amd import wisp
from paper_2606_21868_amd.workloads import WORKLOADS

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_functions():
    names = set()
    for h in sorted(os.listdir(os.path.join(ROOT, "include"))):
        if not h.endswith(".h"):
            continue
        src = open(os.path.join(ROOT, "include", h)).read()
        src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
        names |= set(re.findall(r"\b(wisp_[a-z0-9_]+)\s*\(", src))
    return names


def test_library_exports_every_declared_symbol():
    L = wisp.lib()
    declared = _declared_functions()
    assert len(declared) >= 30
    missing = [n for n in sorted(declared) if not hasattr(L, n)]
    assert not missing, missing
    # the binding covers the whole ABI
    assert declared == set(wisp._SIGS)


def test_exports_are_plain_c_symbols():
    out = os.popen(f"nm -D --defined-only {wisp.LIB_PATH}").read()
    exported = set(re.findall(r"\bT (wisp_[a-z0-9_]+)\b", out))
    assert _declared_functions() <= exported


@pytest.mark.parametrize("name", list(WORKLOADS))
def test_expert_bytes_match_workloads(name):
    wl = WORKLOADS[name]
    assert wisp.expert_bytes(wisp.desc_of(wl)) == wl.blob


def test_invalid_descriptions_rejected_before_any_gpu_call():
    wl = WORKLOADS["tiny-fp32"]
    bad = [
        dict(n_experts=0), dict(n_experts=300), dict(top_k=9), dict(top_k=0), dict(route=7),
        dict(w_dtype=wisp.BF16, x_dtype=wisp.F32), dict(d_model=250), dict(max_tokens=0),
    ]
    for change in bad:
        d = wisp.desc_of(wl)
        for k, v in change.items():
            setattr(d, k, v)
        with pytest.raises(wisp.WispError) as ei:
            wisp.Context(d)
        assert ei.value.status == wisp.E_INVAL, change
        assert wisp.last_error()
    d = wisp.desc_of(WORKLOADS["deepseek-v3-16l-decode"])
    d.n_groups = 7
    with pytest.raises(wisp.WispError):
        wisp.Context(d)


def test_matrix_core_probe_rejects_bad_counts_before_any_gpu_call():
    with pytest.raises(wisp.WispError) as ei:
        wisp.probe_mfma(0)
    assert ei.value.status == wisp.E_INVAL


def test_read_probe_rejects_bad_sizes_before_any_gpu_call():
    for nbytes, launches in ((0, 1), (15, 1), (24, 1), ((1 << 32) + 16, 1), (4096, 0)):
        with pytest.raises(wisp.WispError) as ei:
            wisp.probe_hbm_read(nbytes, launches)
        assert ei.value.status == wisp.E_INVAL, (nbytes, launches)


def _set_trace(rng, N, steps, refs, rho):
    cur = list(rng.choice(N, refs, replace=False))
    out = []
    for _ in range(steps):
        keep = [e for e in cur if rng.random() < rho]
        pool = [e for e in range(N) if e not in keep]
        cur = keep + list(rng.choice(pool, refs - len(keep), replace=False))
        out.append(np.array(cur, np.int32))
    return out


@pytest.mark.parametrize("N,C,T,k,rho", [(128, 32, 1, 8, 0.65), (8, 2, 4, 2, 0.6), (256, 56, 1, 8, 0.7),
                                        (8, 4, 1, 2, 0.5), (16, 3, 2, 4, 0.5), (128, 32, 16, 8, 0.3)])
def test_slot_table_matches_oracle_simulator(N, C, T, k, rho):
    """Two independent implementations of Algorithm 1 (the product's C++ table, the oracle's C
    simulator) agree on hits, misses, chunks, fault lists and slots, step by step."""
    rng = np.random.default_rng(N + 7 * C + T)
    tables = wisp.SlotTable(N, C)
    sim = oracle.LRU(N, C)
    # T tokens' selections per step (duplicates across tokens, as in batched decode)
    for ids in _set_trace(rng, N, 400, min(N, T * k), rho):
        ids = rng.permutation(ids)[: T * k] if T * k <= len(ids) else ids
        sel = np.concatenate([ids, rng.choice(ids, size=max(0, T * k - len(ids)))]).astype(np.int32)
        a = tables.step(sel)
        b = sim.step(sel)
        for key in ("hits", "misses", "chunks"):
            assert a[key] == b[key]
        assert np.array_equal(a["miss_ids"], b["miss_ids"])
        assert np.array_equal(a["miss_slots"], b["miss_slots"])
    for e in range(N):
        assert tables.slot_of(e) == sim.slot(e)


def test_slot_table_resize_matches_oracle():
    rng = np.random.default_rng(3)
    N = 64
    t = wisp.SlotTable(N, 16)
    sim = oracle.LRU(N, 16)
    caps = [16, 9, 9, 30, 4, 64, 1, 12]
    for cap in caps:
        t.resize(cap)
        sim.resize(cap)
        for _ in range(25):
            ids = rng.choice(N, 6, replace=False).astype(np.int32)
            a, b = t.step(ids), sim.step(ids)
            assert (a["hits"], a["misses"], a["chunks"]) == (b["hits"], b["misses"], b["chunks"])
            assert np.array_equal(a["miss_slots"], b["miss_slots"])
        for e in range(N):
            assert t.slot_of(e) == sim.slot(e)
        for s in range(cap):
            assert t.tick(s) == sim.tick(s)
    with pytest.raises(ValueError):
        t.resize(0)
    with pytest.raises(ValueError):
        t.resize(N + 1)
    with pytest.raises(ValueError):
        t.step([N])
    assert wisp.SlotTable(4, 4).cap == 4
    with pytest.raises(ValueError):
        wisp.SlotTable(4, 5)


def test_dit_counts_through_product_slot_table():
    # the paper's DiT-MoE fault counts (Appendix F.1) reproduced by the product's own table
    for cap, want in [(4, (400, 0)), (7, (400, 0)), (8, (8, 392))]:
        t = wisp.SlotTable(8, cap)
        f = h = 0
        for _ in range(50):
            for e in range(8):
                r = t.step([e])
                f += r["misses"]
                h += r["hits"]
        assert (f * 12, h * 12) == (want[0] * 12, want[1] * 12)
