"""GPU parity of the single shared latent (dar_attn_prefill_shared,
dar_cache_append_shared, dar_attn_decode_shared through the C ABI) against
the fp64 oracle: one d_down latent c_j per token and KV head, distant key
c_j U_K, distant value c_j U_V, window keys and values k_j, v_j (Eq. 3-4).
Tolerance: max abs 1e-4 (fp32), 2e-2 (bf16 storage, fp32 accumulation).
"""
import numpy as np
import pytest
import torch

import dar_inputs as di
from oracle import oracle
from tests.dev import to_dev, to_host64, tol

pytestmark = pytest.mark.gpu

dar = pytest.importorskip("paper_2606_18587_amd")

TDT = {"bf16": torch.bfloat16, "f32": torch.float32}


def latents(wl, T, seed):
    """Latents c [B,Hkv,T,dd] ~ N(0,1) and U_K, U_V [Hkv,dd,d] ~ N(0, 1/dd),
    drawn in fp32 and rounded to the workload's dtype."""
    g = np.random.Generator(np.random.PCG64(seed))
    c = di.Tensor(g.standard_normal((wl.B, wl.Hkv, T, wl.dd), dtype=np.float32), wl.dtype)
    uk = di.Tensor(g.standard_normal((wl.Hkv, wl.dd, wl.d), dtype=np.float32) / np.sqrt(wl.dd),
                   wl.dtype)
    uv = di.Tensor(g.standard_normal((wl.Hkv, wl.dd, wl.d), dtype=np.float32) / np.sqrt(wl.dd),
                   wl.dtype)
    return c, uk, uv


def run_prefill(wl, seed=500, check_lse=False):
    inp = di.make_prefill_inputs(wl)
    c, uk, uv = latents(wl, wl.T, seed)
    o, lse = dar.dar_attn_prefill_shared(to_dev(inp["q"]), to_dev(inp["k"]), to_dev(inp["v"]),
                                         to_dev(c), to_dev(uk), to_dev(uv), wl.w, return_lse=True)
    torch.cuda.synchronize()
    got = to_host64(o)
    ref, ref_lse = oracle.prefill_shared(inp["q"].f64, inp["k"].f64, inp["v"].f64, c.f64, uk.f64,
                                         uv.f64, wl.w, want_lse=True)
    assert np.isfinite(got).all()
    err = np.abs(got - ref)
    assert err.max() <= tol(wl.dtype), "max abs err %.3g at %s" % (
        err.max(), np.unravel_index(err.argmax(), err.shape))
    if check_lse:
        assert np.abs(lse.double().cpu().numpy() - ref_lse).max() <= (
            1e-4 if wl.dtype == "f32" else 2e-2)


TINY = di.WORKLOADS["tiny"].with_(B=2, Hq=4, Hkv=2, T=90)
BF16 = di.Workload("shared_bf16", 40, 1, 4, 2, 300, 64, 16, 64, "bf16")


@pytest.mark.parametrize("w", [0, 1, 8, 40, 200])
def test_prefill_fp32_tiny(w):
    run_prefill(TINY.with_(w=w), check_lse=True)


@pytest.mark.parametrize("w", [0, 1, 32, 100, 299, 400])
@pytest.mark.parametrize("d,dd", [(64, 16), (64, 32), (128, 32), (128, 16)])
def test_prefill_bf16_matrix_core(w, d, dd):
    run_prefill(BF16.with_(w=w, d=d, dd=dd), check_lse=(w == 32))


@pytest.mark.parametrize("T", [1, 2, 63, 129, 500])
def test_prefill_bf16_lengths(T):
    run_prefill(BF16.with_(T=T, w=48, B=2))


def test_prefill_bf16_generic_shape():
    run_prefill(di.Workload("shared_generic", 41, 1, 4, 2, 150, 80, 20, 30, "bf16"))


def test_prefill_full_size_every_row():
    """pythia70m shape (B8 H8 T2048 d64 d_down16 w256): every row of every
    head against the oracle (output NaN-filled first)."""
    wl = di.WORKLOADS["pythia70m"]
    inp = di.make_prefill_inputs(wl)
    c, uk, uv = latents(wl, wl.T, 501)
    q = to_dev(inp["q"])
    o = torch.full_like(q, float("nan"))
    dar.dar_attn_prefill_shared(q, to_dev(inp["k"]), to_dev(inp["v"]), to_dev(c), to_dev(uk),
                                to_dev(uv), wl.w, o=o)
    torch.cuda.synchronize()
    got = to_host64(o)
    del q, o
    ref = oracle.prefill_shared(inp["q"].f64, inp["k"].f64, inp["v"].f64, c.f64, uk.f64, uv.f64,
                                wl.w)
    assert np.isfinite(got).all()
    err = np.abs(got - ref).max()
    print("[shared] every row: max abs err %.4g" % err, flush=True)
    assert err <= tol("bf16"), err


# ---------------------------------------------------------------- decode

def raw(x):
    return x.detach().cpu().contiguous().view(
        torch.int16 if x.dtype == torch.bfloat16 else torch.int32).numpy()


def run_decode(wl, L0, steps, seed=510, check_heads=None, bulk=True):
    """Append L0 tokens with their latents, then `steps` x {append one, decode};
    every decode against the oracle's row at position len - 1."""
    pre = di.make_decode_prefix(wl, L0 + steps)
    c, uk, uv = latents(wl, L0 + steps, seed)
    cap = L0 + steps
    cache = dar.DarCache(wl.B, wl.Hkv, wl.d, wl.dd, wl.w, cap, TDT[wl.dtype], shared=True)
    kd, vd, cd = to_dev(pre["k"]), to_dev(pre["v"]), to_dev(c)
    ukd, uvd = to_dev(uk), to_dev(uv)
    if L0 > 0:
        if bulk:
            dar.dar_cache_append_shared(cache, kd[:, :, :L0].contiguous(), vd[:, :, :L0].contiguous(),
                                        cd[:, :, :L0].contiguous(), Hq=wl.Hq)
        else:
            for p in range(L0):
                dar.dar_cache_append_shared(cache, kd[:, :, p:p + 1].contiguous(),
                                            vd[:, :, p:p + 1].contiguous(),
                                            cd[:, :, p:p + 1].contiguous(), Hq=wl.Hq)
    grp = wl.Hq // wl.Hkv
    heads = check_heads or [(b, h) for b in range(wl.B) for h in range(wl.Hq)]
    worst = 0.0
    for t in range(steps):
        p = L0 + t
        dar.dar_cache_append_shared(cache, kd[:, :, p:p + 1].contiguous(), vd[:, :, p:p + 1].contiguous(),
                                    cd[:, :, p:p + 1].contiguous(), Hq=wl.Hq)
        qs = di.make_decode_step(wl, t)["q"]
        o = dar.dar_attn_decode_shared(cache, to_dev(qs), ukd, uvd)
        torch.cuda.synchronize()
        got = to_host64(o)
        assert np.isfinite(got).all()
        L = p + 1
        assert cache.len == L
        for (b, h) in heads:
            g = h // grp
            ref = oracle.rows_shared(pre["k"].f64_slice((b, g))[:L], pre["v"].f64_slice((b, g))[:L],
                                     c.f64_slice((b, g))[:L], uk.f64[g], uv.f64[g], wl.w, [L - 1],
                                     qs.f64[b, h][None])
            worst = max(worst, float(np.abs(got[b, h] - ref[0]).max()))
    assert worst <= tol(wl.dtype), worst
    # the cache holds the given bits: latent slots 0..len-1, ring = newest w tokens
    L = cache.len
    assert np.array_equal(raw(cache.k_lat[:, :, :L]), raw(cd[:, :, :L]))
    for pos in range(max(0, L - wl.w), L):
        assert np.array_equal(raw(cache.k_win[:, :, pos % wl.w]), raw(kd[:, :, pos]))
        assert np.array_equal(raw(cache.v_win[:, :, pos % wl.w]), raw(vd[:, :, pos]))
    return worst


DEC = di.Workload("dec_shared", 42, 2, 8, 2, 0, 64, 16, 32, "bf16", kind="decode")


@pytest.mark.parametrize("w", [0, 1, 32, 600])
def test_decode_bf16(w):
    run_decode(DEC.with_(w=w), 300, 2)


def test_decode_single_token_appends_equal_bulk():
    run_decode(DEC.with_(w=8), 40, 2, bulk=False)


def test_decode_fp32_tiny():
    run_decode(di.Workload("dec_shared_tiny", 43, 1, 2, 2, 0, 16, 4, 8, "f32", kind="decode"), 50, 3)


@pytest.mark.parametrize("G", [1, 2, 8])
def test_decode_group_sizes(G):
    run_decode(DEC.with_(Hq=2 * G, Hkv=2), 130, 2)


@pytest.mark.parametrize("L0,d,dd", [(20000, 64, 16), (9000, 64, 32), (3000, 128, 32),
                                     (2000, 128, 16)])
def test_decode_several_workgroups_per_head(L0, d, dd):
    run_decode(DEC.with_(B=1, d=d, dd=dd, w=256), L0, 2)


def test_decode_matches_prefill_rows():
    """Decoding token p after appending tokens 0..p gives prefill row p."""
    wl = di.Workload("dec_vs_prefill_shared", 44, 1, 4, 2, 160, 64, 16, 24, "bf16")
    inp = di.make_prefill_inputs(wl)
    c, uk, uv = latents(wl, wl.T, 520)
    q, k, v, cd, ukd, uvd = (to_dev(x) for x in (inp["q"], inp["k"], inp["v"], c, uk, uv))
    o_pre = dar.dar_attn_prefill_shared(q, k, v, cd, ukd, uvd, wl.w)
    cache = dar.DarCache(wl.B, wl.Hkv, wl.d, wl.dd, wl.w, wl.T, torch.bfloat16, shared=True)
    worst = 0.0
    for p in range(wl.T):
        dar.dar_cache_append_shared(cache, k[:, :, p:p + 1].contiguous(), v[:, :, p:p + 1].contiguous(),
                                    cd[:, :, p:p + 1].contiguous(), Hq=wl.Hq)
        if p % 13 == 0 or p in (wl.w - 1, wl.w, wl.T - 1):
            o = dar.dar_attn_decode_shared(cache, q[:, :, p].contiguous(), ukd, uvd)
            worst = max(worst, (o.float() - o_pre[:, :, p].float()).abs().max().item())
    torch.cuda.synchronize()
    assert worst <= 2e-2, worst


def test_decode_full_size_sampled_heads():
    """decode1b shape (B32 Hq32 Hkv8 d64 d_down16 w512, 32768 cached tokens)."""
    wl = di.WORKLOADS["decode1b"]
    run_decode(wl, wl.T, 1, check_heads=[(0, 0), (5, 9), (31, 31)])
