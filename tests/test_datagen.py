"""Seeded input generator: Philox known answers, determinism, distributions, encodings."""
import numpy as np
import pytest
import torch

from paper_2606_21868_amd import datagen as dg
from paper_2606_21868_amd.workloads import blob_bytes


# Known-answer vectors for Philox4x32-10 published with the Random123 library (Salmon et al., SC'11).
KAT = [
    ([0, 0, 0, 0], [0, 0], [0x6627E8D5, 0xE169C58D, 0xBC57AC4C, 0x9B00DBD8]),
    ([0xFFFFFFFF] * 4, [0xFFFFFFFF] * 2, [0x408F276D, 0x41C83B0E, 0xA20BC7C6, 0x6D5451FD]),
    ([0x243F6A88, 0x85A308D3, 0x13198A2E, 0x03707344], [0xA4093822, 0x299F31D0],
     [0xD16CFE09, 0x94FDCCEB, 0x5001E420, 0x24126EA1]),
]


@pytest.mark.parametrize("ctr,key,want", KAT)
def test_philox_known_answers(ctr, key, want):
    assert list(dg.philox4x32_10(ctr, key)) == want


def test_normals_deterministic_and_offset_free():
    a = dg.normals(0, dg.KIND_W1, 3, 5, 0, 10_000)
    b = dg.normals(0, dg.KIND_W1, 3, 5, 0, 10_000)
    assert np.array_equal(a, b)
    # any window equals the same slice of a longer run (counter-based, no hidden state)
    for start, n in [(1, 7), (63, 130), (4096, 1000), (9999, 1)]:
        assert np.array_equal(dg.normals(0, dg.KIND_W1, 3, 5, start, n), a[start:start + n])
    # different streams differ
    assert not np.array_equal(a, dg.normals(0, dg.KIND_W1, 3, 6, 0, 10_000))
    assert not np.array_equal(a, dg.normals(1, dg.KIND_W1, 3, 5, 0, 10_000))


def test_normals_distribution():
    from scipy import stats
    z = dg.normals(0, dg.KIND_W2, 0, 0, 0, 400_000).astype(np.float64)
    assert abs(z.mean()) < 0.01
    assert abs(z.var() - 1.0) < 0.01
    assert stats.kstest(z, "norm").pvalue > 1e-3
    # tails: P(|z| > 3) = 0.0027
    assert abs((np.abs(z) > 3).mean() - 0.0027) < 0.0005
    # adjacent elements (same and different Box-Muller pairs) are uncorrelated
    for lag in (1, 2, 4):
        assert abs(np.corrcoef(z[:-lag], z[lag:])[0, 1]) < 0.01


def test_bf16_encoding_matches_torch():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(200_000).astype(np.float32) * 0.02,
                        rng.standard_normal(1000).astype(np.float32) * 1e30,
                        np.array([0.0, -0.0, 1.0, -1.0, 1.00390625, 1.01171875], np.float32)])
    want = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(dg.f32_to_bf16(x), want)


def test_e4m3_encoding_matches_definition():
    # every code's value (torch decodes float8_e4m3fn independently) must encode back to itself
    codes = np.arange(256, dtype=np.uint8)
    vals = torch.from_numpy(codes).view(torch.float8_e4m3fn).float().numpy()
    finite = ~np.isnan(vals)
    got = dg.f32_to_e4m3(vals[finite])
    want = codes[finite].copy()
    want[want == 0x80] = 0x80  # -0 stays -0
    assert np.array_equal(got, want)
    # round to nearest even against torch for in-range values (torch does not saturate)
    rng = np.random.default_rng(1)
    x = np.concatenate([rng.standard_normal(300_000) * s for s in (0.001, 0.05, 3.0, 100.0)]).astype(np.float32)
    x = np.clip(x, -448, 448)
    want = torch.from_numpy(x).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(dg.f32_to_e4m3(x), want)
    # exact halfway points between neighbouring codes round to the even code
    pos = vals[(codes < 0x7E) & finite & (vals >= 0)]
    mids = ((pos[:-1].astype(np.float64) + pos[1:]) / 2).astype(np.float32)
    got = dg.f32_to_e4m3(mids)
    lo = np.arange(len(mids))
    even = np.where(lo % 2 == 0, lo, lo + 1)
    assert np.array_equal(got, even.astype(np.uint8))
    # saturation
    assert dg.f32_to_e4m3(np.array([448.0, 449.0, 1e6, -1e6], np.float32)).tolist() == [0x7E, 0x7E, 0x7E, 0xFE]


@pytest.mark.parametrize("dtype,d,I", [(dg.F32, 256, 512), (dg.BF16, 2048, 768), (dg.FP8, 256, 384)])
def test_blob_layout(dtype, d, I):
    b = dg.expert_blob(0, 2, 7, dtype, d, I)
    assert b.size == dg.blob_bytes(dtype, d, I) == blob_bytes(dtype, d, I)
    n = d * I
    if dtype == dg.F32:
        w = b.view(np.float32)
        w1 = w[:n].reshape(I, d)
        assert np.array_equal(w1[1], np.float32(0.02) * dg.normals(0, dg.KIND_W1, 2, 7, d, d))
        w2 = w[2 * n:].reshape(d, I)
        assert np.array_equal(w2[3], np.float32(0.02) * dg.normals(0, dg.KIND_W2, 2, 7, 3 * I, I))
    elif dtype == dg.BF16:
        w = b.view(np.uint16)
        w3 = w[n:2 * n].reshape(I, d)
        assert np.array_equal(w3[5], dg.f32_to_bf16(np.float32(0.02) * dg.normals(0, dg.KIND_W3, 2, 7, 5 * d, d)))
    else:
        q = b[:3 * n]
        sc = b[3 * n:].view(np.uint16)
        assert sc.size == 3 * (d // 128) * (I // 128)
        # decoded weights approximate 0.02 z within half a quantum of each block
        w1 = torch.from_numpy(q[:n].copy()).view(torch.float8_e4m3fn).float().numpy().reshape(I, d)
        s1 = torch.from_numpy(sc[:(I // 128) * (d // 128)].copy().view(np.int16)).view(torch.bfloat16).float()
        s1 = s1.numpy().reshape(I // 128, d // 128)
        dec = w1 * np.repeat(np.repeat(s1, 128, 0), 128, 1)
        ref = np.float32(0.02) * dg.normals(0, dg.KIND_W1, 2, 7, 0, n).reshape(I, d)
        rel = np.abs(dec - ref) / np.repeat(np.repeat(s1 * 448, 128, 0), 128, 1)
        assert rel.max() < 2 ** -4
        # every block uses its range: the block's amax code is near 448 (scale is bf16-rounded)
        assert np.abs(w1).max() >= 400


def test_blobs_parallel_equals_single():
    ptr_arrays = [np.zeros(dg.blob_bytes(dg.BF16, 256, 384), np.uint8) for _ in range(5)]
    dg.fill_blobs(0, [0, 0, 1, 1, 2], [0, 3, 0, 3, 4095], [a.ctypes.data for a in ptr_arrays], dg.BF16, 256, 384,
                  threads=4)
    for a, (l, e) in zip(ptr_arrays, [(0, 0), (0, 3), (1, 0), (1, 3), (2, 4095)]):
        assert np.array_equal(a, dg.expert_blob(0, l, e, dg.BF16, 256, 384))


def test_ar1_states():
    x = dg.decode_inputs(0, L=2, S=400, T=3, d=512, dtype=dg.F32).astype(np.float64)
    # x_0 = eps_0 and the recursion in fp64 (stored via fp32)
    eps0 = dg.normals(0, dg.KIND_XAR, 1, 2, 0, 512)
    assert np.array_equal(x[1, 0, 2], eps0.astype(np.float32).astype(np.float64))
    # stationary unit variance and lag-1 autocorrelation rho = 0.9
    v = x.var()
    assert abs(v - 1.0) < 0.05
    r1 = (x[:, 1:] * x[:, :-1]).mean() / v
    assert abs(r1 - 0.9) < 0.02
    # chains of different layers / rows are independent
    assert abs(np.corrcoef(x[0, :, 0].ravel(), x[1, :, 0].ravel())[0, 1]) < 0.05
    xb = dg.decode_inputs(0, L=2, S=10, T=3, d=512, dtype=dg.BF16)
    assert xb.dtype == np.uint16
    assert np.array_equal(xb[0, 3, 1], dg.f32_to_bf16(dg.decode_inputs(0, 2, 10, 3, 512, dg.F32)[0, 3, 1]))


def test_router_weights_scale():
    w = dg.router_weights(0, 0, 128, 2048)
    assert abs(w.std() * np.sqrt(2048) - 1.0) < 0.01
