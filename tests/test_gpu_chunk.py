"""GPU chunked prefill (dar_attn_prefill_chunk through the C ABI).

A cache holding the first L tokens of a sequence takes the next n tokens in
one call. Checked against what the method fixes for those rows and that
cache:
  * the n outputs equal rows L..L+n-1 of the oracle's prefill over the whole
    sequence 0..L+n-1 (Eq. 3-4; tolerance as for prefill: 1e-4 fp32, 2e-2
    bf16 with fp32 accumulation), element by element;
  * the cache afterwards is byte-identical to appending the same n tokens
    with dar_cache_append (ring slots and latents);
  * a sequence fed as several chunks gives every row of the whole-sequence
    prefill.
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


def raw(x):
    return x.detach().cpu().contiguous().view(
        torch.int16 if x.dtype == torch.bfloat16 else torch.int32).numpy()


def append_all(wl, kd, vd, wdd, cap, chunks):
    c = dar.DarCache(wl.B, wl.Hkv, wl.d, wl.dd, wl.w, cap, TDT[wl.dtype])
    pos = 0
    for ch in chunks:
        dar.dar_cache_append(c, kd[:, :, pos:pos + ch].contiguous(),
                             vd[:, :, pos:pos + ch].contiguous(), wdd, Hq=wl.Hq)
        pos += ch
    return c


def same_cache(a, b):
    assert a.len == b.len
    if a.w > 0:
        assert np.array_equal(raw(a.k_win), raw(b.k_win)), "ring keys differ"
        assert np.array_equal(raw(a.v_win), raw(b.v_win)), "ring values differ"
    n_lat = max(0, a.len - a.w)
    assert np.array_equal(raw(a.k_lat[:, :, :n_lat]), raw(b.k_lat[:, :, :n_lat])), "latent keys differ"
    assert np.array_equal(raw(a.v_lat[:, :, :n_lat]), raw(b.v_lat[:, :, :n_lat])), "latent values differ"


def run_chunks(wl, chunks, untied=False, prefix=None, check_lse=False):
    """Feed the sequence: the first `prefix` tokens by dar_cache_append (as a
    cache would hold them), then each chunk by dar_attn_prefill_chunk.
    Returns the max abs error of all chunked rows against the oracle."""
    inp = di.make_prefill_inputs(wl, untied=untied)
    q, kd, vd = to_dev(inp["q"]), to_dev(inp["k"]), to_dev(inp["v"])
    wdd, wud = to_dev(inp["wd"]), to_dev(inp["wu"])
    ref, ref_lse = oracle.prefill(inp["q"].f64, inp["k"].f64, inp["v"].f64, inp["wd"].f64,
                                  None if inp["wu"] is None else inp["wu"].f64, wl.w,
                                  want_lse=True)
    cap = wl.T + 3
    pre = list(prefix or [])
    c = append_all(wl, kd, vd, wdd, cap, pre)
    pos = sum(pre)
    worst = 0.0
    for n in chunks:
        sl = slice(pos, pos + n)
        o, lse = dar.dar_attn_prefill_chunk(c, q[:, :, sl].contiguous(), kd[:, :, sl].contiguous(),
                                            vd[:, :, sl].contiguous(), wdd, wud, return_lse=True)
        torch.cuda.synchronize()
        got = to_host64(o)
        assert np.isfinite(got).all()
        err = np.abs(got - ref[:, :, sl])
        assert err.max() <= tol(wl.dtype), "chunk at %d (+%d): max abs err %.3g at %s" % (
            pos, n, err.max(), np.unravel_index(err.argmax(), err.shape))
        if check_lse:
            lerr = np.abs(lse.double().cpu().numpy() - ref_lse[:, :, sl]).max()
            assert lerr <= (1e-4 if wl.dtype == "f32" else 2e-2), lerr
        worst = max(worst, float(err.max()))
        pos += n
        assert c.len == pos
    assert pos == wl.T
    same_cache(c, append_all(wl, kd, vd, wdd, cap, [wl.T]))
    return worst


TINY = di.WORKLOADS["tiny"].with_(B=2, Hq=4, Hkv=2)   # fp32 d16 d_down4


@pytest.mark.parametrize("w", [0, 1, 8, 40])
@pytest.mark.parametrize("L,n", [(0, 37), (5, 1), (30, 17), (50, 50)])
def test_fp32_chunk_after_prefix(w, L, n):
    run_chunks(TINY.with_(w=w, T=L + n), [n], untied=(w % 2 == 1), prefix=[L] if L else None)


BF16 = di.Workload("chunk_bf16", 20, 2, 4, 2, 0, 64, 16, 32, "bf16")


@pytest.mark.parametrize("w", [0, 1, 32, 100, 400])
@pytest.mark.parametrize("L,n", [(0, 150), (37, 1), (200, 64), (300, 129), (250, 333)])
def test_bf16_d64_chunk_after_prefix(w, L, n):
    run_chunks(BF16.with_(w=w, T=L + n), [n], untied=(w == 100), prefix=[L] if L else None)


@pytest.mark.parametrize("wl,L,n,untied", [
    (di.Workload("chunk_d128", 21, 1, 8, 2, 0, 128, 32, 64, "bf16"), 257, 190, True),
    (di.Workload("chunk_d64_32", 22, 1, 4, 4, 0, 64, 32, 48, "bf16"), 130, 70, False),
    (di.Workload("chunk_generic", 23, 1, 2, 1, 0, 80, 20, 24, "bf16"), 90, 41, False),
    # d 64 with d_down 8: the pre-pass and the appends must take the same
    # (vector-ALU) projection for the cache to be byte-equal to appends
    (di.Workload("chunk_d64_dd8", 25, 1, 4, 2, 0, 64, 8, 40, "bf16"), 150, 60, False),
])
def test_other_shapes(wl, L, n, untied):
    run_chunks(wl.with_(T=L + n), [n], untied=untied, prefix=[L], check_lse=True)


@pytest.mark.parametrize("wl,chunks", [
    (TINY.with_(w=8, T=70), [20, 1, 30, 19]),
    (BF16.with_(w=64, T=600), [100, 1, 250, 249]),
    (BF16.with_(w=0, T=300), [128, 128, 44]),
    (BF16.with_(w=512, T=700), [300, 300, 100]),
])
def test_sequence_in_chunks(wl, chunks):
    """Every row of a whole-sequence prefill, computed chunk by chunk from an
    empty cache; the first chunk is a plain prefill."""
    run_chunks(wl, chunks)


def test_chunk_of_one_equals_decode():
    """A one-token chunk is a decode step: its row equals dar_attn_decode after
    appending the token (the same query at position len - 1)."""
    wl = BF16.with_(w=48, T=301)
    inp = di.make_prefill_inputs(wl)
    q, kd, vd, wdd = to_dev(inp["q"]), to_dev(inp["k"]), to_dev(inp["v"]), to_dev(inp["wd"])
    c1 = append_all(wl, kd, vd, wdd, wl.T, [wl.T - 1])
    c2 = append_all(wl, kd, vd, wdd, wl.T, [wl.T])
    sl = slice(wl.T - 1, wl.T)
    oc = dar.dar_attn_prefill_chunk(c1, q[:, :, sl].contiguous(), kd[:, :, sl].contiguous(),
                                    vd[:, :, sl].contiguous(), wdd)
    od = dar.dar_attn_decode(c2, q[:, :, wl.T - 1].contiguous(), wdd)
    torch.cuda.synchronize()
    assert np.abs(to_host64(oc[:, :, 0]) - to_host64(od)).max() <= tol(wl.dtype)
    same_cache(c1, c2)


def test_full_size_every_row():
    """A long cache (8192 tokens, window 512) and a 1024-token chunk: every
    row of every head against the oracle's evaluation over the whole history
    (output NaN-filled first)."""
    wl = di.Workload("chunk_long", 24, 2, 8, 2, 9216, 64, 16, 512, "bf16")
    L, n = 8192, 1024
    inp = di.make_prefill_inputs(wl)
    q, kd, vd, wdd = to_dev(inp["q"]), to_dev(inp["k"]), to_dev(inp["v"]), to_dev(inp["wd"])
    c = append_all(wl, kd, vd, wdd, wl.T, [L])
    sl = slice(L, L + n)
    o = torch.full((wl.B, wl.Hq, n, wl.d), float("nan"), dtype=q.dtype, device=q.device)
    dar.dar_attn_prefill_chunk(c, q[:, :, sl].contiguous(), kd[:, :, sl].contiguous(),
                               vd[:, :, sl].contiguous(), wdd, o=o)
    torch.cuda.synchronize()
    got = to_host64(o)
    assert np.isfinite(got).all()
    grp = wl.Hq // wl.Hkv
    rows = np.arange(L, L + n)
    worst = 0.0
    for b in range(wl.B):
        for g in range(wl.Hkv):
            hs = list(range(g * grp, (g + 1) * grp))
            qr = inp["q"].f64[b, hs][:, L:L + n].reshape(-1, wl.d)
            ref = oracle.rows(inp["k"].f64[b, g], inp["v"].f64[b, g], inp["wd"].f64[g], None, wl.w,
                              np.tile(rows, grp), qr)
            worst = max(worst, float(np.abs(got[b, hs].reshape(-1, wl.d) - ref).max()))
    print("[chunk] every row: max abs err %.4g" % worst, flush=True)
    assert worst <= tol(wl.dtype), worst
