"""Split-cache exactness on the GPU (dar_cache_append through the C ABI).

Bit-exact: which token sits in which ring slot and latent slot, bulk appends
against single-token appends, and latents of a selection-matrix W_down
(exact copies of the first d_down key/value coordinates). Latent values for a
random W_down are compared with the oracle's Eq. 1 within bf16 rounding.
"""
import numpy as np
import pytest
import torch

import dar_inputs as di
from oracle import oracle
from tests.dev import to_dev, to_host64

pytestmark = pytest.mark.gpu

dar = pytest.importorskip("paper_2606_18587_amd")


def tokens(B, Hkv, n, d, dtype, seed):
    g = np.random.Generator(np.random.PCG64(seed))
    k = di.Tensor(g.standard_normal((B, Hkv, n, d), dtype=np.float32), dtype)
    v = di.Tensor(g.standard_normal((B, Hkv, n, d), dtype=np.float32), dtype)
    return k, v


def wdown(Hkv, d, dd, dtype, seed, selection=False):
    if selection:
        w = np.zeros((Hkv, d, dd), np.float32)
        for g in range(Hkv):
            w[g, :dd, :] = np.eye(dd)
        return di.Tensor(w, dtype)
    g = np.random.Generator(np.random.PCG64(seed))
    return di.Tensor(g.standard_normal((Hkv, d, dd), dtype=np.float32) / np.sqrt(d), dtype)


TDT = {"bf16": torch.bfloat16, "f32": torch.float32}


def build(k, v, wd, w, cap, chunks, dd):
    B, Hkv, n, d = k.shape
    c = dar.DarCache(B, Hkv, d, dd, w, cap, TDT[k.dtype])
    kd, vd, wdd = to_dev(k), to_dev(v), to_dev(wd)
    pos = 0
    for ch in chunks:
        dar.dar_cache_append(c, kd[:, :, pos:pos + ch].contiguous(),
                             vd[:, :, pos:pos + ch].contiguous(), wdd)
        pos += ch
    assert pos == n and c.len == n
    torch.cuda.synchronize()
    return c


def raw(x):
    return x.detach().cpu().contiguous().view(torch.int16 if x.dtype == torch.bfloat16 else torch.int32).numpy()


def check_slots(c, k, v, n, w):
    ring, lat = oracle.cache_model(n, w, c.cap)
    kr, vr = raw(c.k_win), raw(c.v_win)
    ks = k.store.view(np.int16 if k.dtype == "bf16" else np.int32)
    vs = v.store.view(np.int16 if v.dtype == "bf16" else np.int32)
    for s, p in enumerate(ring):
        if p >= 0:
            assert np.array_equal(kr[:, :, s], ks[:, :, p]), (s, p)
            assert np.array_equal(vr[:, :, s], vs[:, :, p]), (s, p)
    return lat


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("w,n,chunks", [
    (8, 50, [50]),                 # bulk, n > w (two-phase append)
    (8, 50, [1] * 50),             # single-token appends
    (8, 50, [3, 8, 1, 20, 7, 11]),  # chunks around the window size
    (16, 10, [10]),                # never leaves the window
    (16, 16, [16]),                # fills it exactly
    (0, 30, [30]),                 # no window: every token goes to the latents
    (0, 30, [1] * 30),
    (64, 200, [64, 64, 72]),
])
def test_selection_matrix_latents_and_ring_slots(dtype, w, n, chunks):
    B, Hkv, d, dd = 2, 3, 64, 16
    k, v = tokens(B, Hkv, n, d, dtype, 1234 + n + w)
    wd = wdown(Hkv, d, dd, dtype, 0, selection=True)
    c = build(k, v, wd, w, 256, chunks, dd)
    lat = check_slots(c, k, v, n, w)
    ne = int(lat.sum())
    kl, vl = raw(c.k_lat), raw(c.v_lat)
    ks = k.store.view(np.int16 if dtype == "bf16" else np.int32)
    vs = v.store.view(np.int16 if dtype == "bf16" else np.int32)
    assert np.array_equal(kl[:, :, :ne], ks[:, :, :ne, :dd])
    assert np.array_equal(vl[:, :, :ne], vs[:, :, :ne, :dd])
    assert not kl[:, :, ne:].any() and not vl[:, :, ne:].any()   # untouched slots stay zero


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("w", [0, 5, 32])
def test_bulk_equals_incremental(dtype, w):
    B, Hkv, d, dd, n = 2, 2, 64, 16, 120
    k, v = tokens(B, Hkv, n, d, dtype, 99 + w)
    wd = wdown(Hkv, d, dd, dtype, 7)
    a = build(k, v, wd, w, 128, [n], dd)
    b = build(k, v, wd, w, 128, [1] * n, dd)
    cc = build(k, v, wd, w, 128, [13, 1, 40, 2, 64], dd)
    for x in ("k_win", "v_win", "k_lat", "v_lat"):
        assert np.array_equal(raw(getattr(a, x)), raw(getattr(b, x))), x
        assert np.array_equal(raw(getattr(a, x)), raw(getattr(cc, x))), x


@pytest.mark.parametrize("dtype,d,dd", [("bf16", 64, 16), ("bf16", 128, 32), ("f32", 16, 4)])
def test_latent_values_match_eq1(dtype, d, dd):
    B, Hkv, n, w = 2, 2, 90, 10
    k, v = tokens(B, Hkv, n, d, dtype, 5)
    wd = wdown(Hkv, d, dd, dtype, 6)
    c = build(k, v, wd, w, 100, [n], dd)
    got_k = to_host64(c.k_lat)[:, :, : n - w]
    got_v = to_host64(c.v_lat)[:, :, : n - w]
    for b in range(B):
        for g in range(Hkv):
            ref_k = oracle.down(k.f64[b, g, : n - w], wd.f64[g])
            ref_v = oracle.down(v.f64[b, g, : n - w], wd.f64[g])
            # one rounding to the cache dtype
            rel = 2.0 ** -8 if dtype == "bf16" else 1e-6
            assert np.all(np.abs(got_k[b, g] - ref_k) <= rel * np.abs(ref_k) + 1e-6)
            assert np.all(np.abs(got_v[b, g] - ref_v) <= rel * np.abs(ref_v) + 1e-6)


def test_capacity_error_leaves_cache_unchanged():
    B, Hkv, d, dd, w = 1, 2, 64, 16, 4
    k, v = tokens(B, Hkv, 20, d, "bf16", 3)
    wd = wdown(Hkv, d, dd, "bf16", 4)
    c = build(k, v, wd, w, 24, [20], dd)
    before = [raw(getattr(c, x)).copy() for x in ("k_win", "v_win", "k_lat", "v_lat")]
    extra_k, extra_v = tokens(B, Hkv, 5, d, "bf16", 8)
    with pytest.raises(dar.DarError) as ei:
        dar.dar_cache_append(c, to_dev(extra_k), to_dev(extra_v), to_dev(wd))
    assert ei.value.status == dar.DAR_E_CAPACITY
    torch.cuda.synchronize()
    assert c.len == 20
    after = [raw(getattr(c, x)) for x in ("k_win", "v_win", "k_lat", "v_lat")]
    for a, b in zip(before, after):
        assert np.array_equal(a, b)
