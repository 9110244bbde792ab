"""GPU chunked prefill with the rotary embedding of Eq. 3
(dar_attn_prefill_chunk_rope through the C ABI).

A cache holding the first L tokens of a sequence (un-rotated, as
dar_cache_append stores them) takes the next n tokens in one call, with the
rotation where Eq. 3 puts it: window keys rotated at their positions, distant
keys lifted and then rotated (those below L - w from the cache's latents).
Checked against what the method fixes for those rows and that cache:
  * the n outputs and their log-sum-exp equal rows L..L+n-1 of the oracle's
    rotary prefill over the whole sequence 0..L+n-1 (tolerance 2e-2 for bf16
    with fp32 accumulation), element by element;
  * the cache afterwards is byte-identical to appending the same n tokens with
    dar_cache_append;
  * a sequence fed as several chunks gives every row of the whole-sequence
    rotary prefill, and a rotary decode step after the chunks gives the
    oracle's row at the next position.
"""
import numpy as np
import pytest
import torch

import dar_inputs as di
from oracle import oracle
from tests.dev import to_dev, to_host64, tol

pytestmark = pytest.mark.gpu

dar = pytest.importorskip("paper_2606_18587_amd")


def raw(x):
    return x.detach().cpu().contiguous().view(torch.int16).numpy()


def append_all(wl, kd, vd, wdd, cap, chunks):
    c = dar.DarCache(wl.B, wl.Hkv, wl.d, wl.dd, wl.w, cap, torch.bfloat16)
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


def run_chunks(wl, chunks, r, base=10000.0, untied=False, prefix=0, decode_after=False):
    """The first `prefix` tokens by dar_cache_append, then each chunk by
    dar_attn_prefill_chunk_rope; every chunked row against the oracle's rotary
    prefill of the whole sequence. Returns the largest abs error."""
    T = prefix + sum(chunks)
    wl = wl.with_(T=T)
    inp = di.make_prefill_inputs(wl, untied=untied)
    q, kd, vd = to_dev(inp["q"]), to_dev(inp["k"]), to_dev(inp["v"])
    wdd, wud = to_dev(inp["wd"]), to_dev(inp["wu"])
    wu64 = None if inp["wu"] is None else inp["wu"].f64
    ref, ref_lse = oracle.prefill_rope(inp["q"].f64, inp["k"].f64, inp["v"].f64, inp["wd"].f64, wu64,
                                       wl.w, r, base, 0, want_lse=True)
    cap = T + 2
    rope = dar.Rope(r, base, n_pos=cap)
    c = append_all(wl, kd, vd, wdd, cap, [prefix] if prefix else [])
    pos = prefix
    worst = 0.0
    for n in chunks:
        sl = slice(pos, pos + n)
        o = torch.full((wl.B, wl.Hq, n, wl.d), float("nan"), dtype=torch.bfloat16, device="cuda")
        lse = torch.full((wl.B, wl.Hq, n), float("nan"), dtype=torch.float32, device="cuda")
        dar.dar_attn_prefill_chunk_rope(c, q[:, :, sl].contiguous(), kd[:, :, sl].contiguous(),
                                        vd[:, :, sl].contiguous(), wdd, rope, w_up=wud, o=o, lse=lse)
        torch.cuda.synchronize()
        got = to_host64(o)
        assert np.isfinite(got).all()
        err = np.abs(got - ref[:, :, sl])
        assert err.max() <= tol("bf16"), "chunk at %d (+%d): max abs err %.3g at %s" % (
            pos, n, err.max(), np.unravel_index(err.argmax(), err.shape))
        lerr = np.abs(lse.double().cpu().numpy() - ref_lse[:, :, sl]).max()
        assert lerr <= 2e-2, lerr
        worst = max(worst, float(err.max()))
        pos += n
        assert c.len == pos
    same_cache(c, append_all(wl, kd, vd, wdd, cap, [T]))
    if decode_after:
        # one more token, then a rotary decode at position T against the oracle
        g = np.random.Generator(np.random.PCG64(90))
        kn = di.Tensor(g.standard_normal((wl.B, wl.Hkv, 1, wl.d), dtype=np.float32), "bf16")
        vn = di.Tensor(g.standard_normal((wl.B, wl.Hkv, 1, wl.d), dtype=np.float32), "bf16")
        qn = di.Tensor(g.standard_normal((wl.B, wl.Hq, wl.d), dtype=np.float32), "bf16")
        dar.dar_cache_append(c, to_dev(kn), to_dev(vn), wdd, Hq=wl.Hq)
        od = to_host64(dar.dar_attn_decode_rope(c, to_dev(qn), wdd, rope, w_up=wud))
        grp = wl.Hq // wl.Hkv
        for b in range(wl.B):
            for h in range(wl.Hq):
                gg = h // grp
                K = np.concatenate([inp["k"].f64[b, gg], kn.f64[b, gg]])
                V = np.concatenate([inp["v"].f64[b, gg], vn.f64[b, gg]])
                row = oracle.rows_rope(K, V, inp["wd"].f64[gg], None if wu64 is None else wu64[gg],
                                       wl.w, r, base, 0, [T], qn.f64[b, h][None])
                assert np.abs(od[b, h] - row[0]).max() <= tol("bf16")
    return worst


D64 = di.Workload("chunk_rope", 26, 2, 4, 2, 0, 64, 16, 32, "bf16")


@pytest.mark.parametrize("w", [0, 32, 100])
@pytest.mark.parametrize("L,n", [(0, 70), (5, 1), (45, 30), (200, 64), (37, 140)])
@pytest.mark.parametrize("r", [16, 64])
def test_chunk_rope_after_prefix(w, L, n, r):
    run_chunks(D64.with_(w=w), [n], r, untied=(w == 100), prefix=L)


@pytest.mark.parametrize("w,L,n,r,untied", [(64, 100, 40, 32, False), (64, 0, 97, 128, True),
                                            (200, 333, 65, 64, False), (0, 90, 33, 16, True)])
def test_chunk_rope_d128(w, L, n, r, untied):
    run_chunks(di.Workload("chunk_rope_d128", 27, 1, 8, 2, 0, 128, 32, w, "bf16"), [n], r,
               base=500000.0, untied=untied, prefix=L)


def test_chunk_rope_several_chunks_then_decode():
    """A sequence as chunks of uneven sizes (window 48: the context start
    moves across 32-row blocks between calls), then a rotary decode step on
    the cache the chunks left."""
    run_chunks(D64.with_(w=48), [50, 31, 64, 1, 97], 32, decode_after=True)


def test_chunk_rope_d_down_32():
    run_chunks(di.Workload("chunk_rope_dd32", 28, 1, 4, 4, 0, 64, 32, 80, "bf16"), [60, 70], 64,
               untied=True, prefix=130)


def test_chunk_rope_full_size_pythia70m():
    """The pythia70m shape (B8 H8 d64 d_down16 w256, 2048 positions): its
    last 256 tokens as one chunk into a cache of the first 1792, rotary
    dimension 16 of the Pythia models."""
    wl = di.WORKLOADS["pythia70m"]
    run_chunks(wl, [256], 16, prefix=wl.T - 256)
