"""GPU parity of the rotary embedding inside Eq. 3 (dar_rope_table,
dar_attn_prefill_rope through the C ABI) against the fp64 oracle.

The queries and keys handed over are un-rotated; the window keys are rotated
at their positions, the distant keys after the lift, values never (Eq. 3).
Tolerance as for prefill: max abs 1e-4 (fp32), 2e-2 (bf16 storage, fp32
accumulation), element by element.
"""
import numpy as np
import pytest
import torch

import dar_inputs as di
from oracle import oracle
from tests.dev import to_dev, to_host64, tol

pytestmark = pytest.mark.gpu

dar = pytest.importorskip("paper_2606_18587_amd")


@pytest.mark.parametrize("r,base,n_pos", [(64, 10000.0, 4096), (16, 10000.0, 33000),
                                          (128, 500000.0, 70), (2, 10.0, 5)])
def test_table_matches_oracle(r, base, n_pos):
    """Each entry is the fp64 cos/sin rounded to fp32 (at most one fp32 step
    apart where the two fp64 libraries round a value differently)."""
    got = dar.dar_rope_table(r, base, n_pos).cpu().numpy().astype(np.float64)
    ref = oracle.rope_table(r, base, n_pos)
    step = np.spacing(np.abs(ref).astype(np.float32)).astype(np.float64)
    assert (np.abs(got - ref) <= step).all()


def run(wl, r, base, pos0=0, untied=False, check_lse=False, q_scale=1.0):
    inp = di.make_prefill_inputs(wl, untied=untied, q_scale=q_scale)
    q, k, v = to_dev(inp["q"]), to_dev(inp["k"]), to_dev(inp["v"])
    wd, wu = to_dev(inp["wd"]), to_dev(inp["wu"])
    rope = dar.Rope(r, base, n_pos=pos0 + wl.T)
    o, lse = dar.dar_attn_prefill_rope(q, k, v, wd, wu, wl.w, rope, pos0=pos0, return_lse=True)
    torch.cuda.synchronize()
    got = to_host64(o)
    ref, ref_lse = oracle.prefill_rope(inp["q"].f64, inp["k"].f64, inp["v"].f64, inp["wd"].f64,
                                       None if inp["wu"] is None else inp["wu"].f64, wl.w, r, base,
                                       pos0=pos0, want_lse=True)
    assert np.isfinite(got).all()
    err = np.abs(got - ref)
    assert err.max() <= tol(wl.dtype), "max abs err %.3g at %s" % (
        err.max(), np.unravel_index(err.argmax(), err.shape))
    if check_lse:
        lerr = np.abs(lse.double().cpu().numpy() - ref_lse).max()
        assert lerr <= (1e-4 if wl.dtype == "f32" else 2e-2), lerr
    return float(err.max())


TINY = di.WORKLOADS["tiny"].with_(B=2, Hq=4, Hkv=2, T=90)   # fp32 d16 d_down4


@pytest.mark.parametrize("w", [0, 1, 8, 40, 200])
@pytest.mark.parametrize("r,pos0", [(16, 0), (8, 37), (0, 5), (2, 1000)])
def test_fp32_tiny(w, r, pos0):
    run(TINY.with_(w=w), r, 10000.0, pos0=pos0, untied=(w % 2 == 1), check_lse=True)


BF16 = di.Workload("rope_bf16", 30, 1, 4, 2, 300, 64, 16, 64, "bf16")


@pytest.mark.parametrize("w", [0, 1, 32, 100, 299, 400])
@pytest.mark.parametrize("r,base", [(64, 10000.0), (16, 10000.0), (32, 500000.0)])
def test_bf16_d64_matrix_core(w, r, base):
    run(BF16.with_(w=w), r, base, untied=(w == 100), check_lse=(w == 32))


@pytest.mark.parametrize("T", [1, 2, 63, 129, 257, 500])
def test_bf16_d64_lengths(T):
    run(BF16.with_(T=T, w=48, B=2), 64, 10000.0, pos0=3)


@pytest.mark.parametrize("w,r", [(0, 128), (64, 128), (100, 32), (512, 64)])
def test_bf16_d128_gqa(w, r):
    run(di.Workload("rope_d128", 31, 1, 8, 2, 400, 128, 32, w, "bf16"), r, 500000.0,
        untied=(w == 100), check_lse=True)


@pytest.mark.parametrize("d,dd,w,T,r", [(80, 20, 30, 150, 80), (48, 12, 10, 90, 16),
                                        (64, 64, 20, 120, 64), (128, 8, 50, 170, 64)])
def test_bf16_other_shapes(d, dd, w, T, r):
    """d not in {64, 128} takes the generic kernels; any d_down works on the
    matrix-core path (the lift happens before the attention)."""
    run(di.Workload("rope_other", 32, 1, 4, 2, T, d, dd, w, "bf16"), r, 10000.0, untied=True)


def test_large_positions():
    """Positions near 33K (a long cache): large angles."""
    run(BF16.with_(T=200, w=40), 64, 10000.0, pos0=32700)


def test_peaky_queries():
    """Queries scaled by 2 (sharper rows). The rotated query and key are
    rounded to bf16 before the matrix cores multiply them (the operands the
    rotation-free path takes exactly as given), an error proportional to
    the score size: measured 0.012 at unit scale, 0.014 here, 0.032 at x4
    (the rotation-free path: 0.015 at x4)."""
    run(BF16.with_(w=64, T=400), 64, 10000.0, q_scale=2.0)


def test_shift_invariance_on_gpu():
    """Scores depend on positions only through i - j: moving the whole
    sequence changes the output by rounding only."""
    wl = BF16.with_(w=50, T=260)
    inp = di.make_prefill_inputs(wl)
    q, k, v, wd = to_dev(inp["q"]), to_dev(inp["k"]), to_dev(inp["v"]), to_dev(inp["wd"])
    rope = dar.Rope(64, 10000.0, n_pos=5000)
    a = dar.dar_attn_prefill_rope(q, k, v, wd, None, wl.w, rope, pos0=0)
    b = dar.dar_attn_prefill_rope(q, k, v, wd, None, wl.w, rope, pos0=4000)
    torch.cuda.synchronize()
    assert np.abs(to_host64(a) - to_host64(b)).max() <= tol("bf16")


@pytest.mark.parametrize("r,base", [(16, 10000.0), (64, 500000.0)])
def test_full_size_every_row(r, base):
    """The pythia70m-shaped prefill (B8 H8 T2048 d64 d_down16 w256) with the
    Pythia rotary fraction (16 of 64 dims) and with full rotation: every row
    of every head against the oracle (output NaN-filled first)."""
    wl = di.WORKLOADS["pythia70m"]
    inp = di.make_prefill_inputs(wl)
    q, k, v, wd = to_dev(inp["q"]), to_dev(inp["k"]), to_dev(inp["v"]), to_dev(inp["wd"])
    rope = dar.Rope(r, base, n_pos=wl.T)
    o = torch.full_like(q, float("nan"))
    dar.dar_attn_prefill_rope(q, k, v, wd, None, wl.w, rope, o=o)
    torch.cuda.synchronize()
    got = to_host64(o)
    del q, k, v, o
    ref = oracle.prefill_rope(inp["q"].f64, inp["k"].f64, inp["v"].f64, inp["wd"].f64, None, wl.w,
                              r, base)
    assert np.isfinite(got).all()
    err = np.abs(got - ref).max()
    print("[rope r=%d] every row: max abs err %.4g" % (r, err), flush=True)
    assert err <= tol("bf16"), err


# ---------------------------------------------------------------- decode

TDT = {"bf16": torch.bfloat16, "f32": torch.float32}


def run_decode_rope(wl, L0, steps, r, base=10000.0, untied=False, check_heads=None):
    """Append L0 tokens, then `steps` x {append one, decode with RoPE}; each
    decode against the oracle's row at position len - 1 (RoPE inside Eq. 3
    over the full-dimension history, tokens at positions 0..len-1)."""
    pre = di.make_decode_prefix(wl, L0)
    wd = pre["wd"]
    wu = None
    if untied:
        g = np.random.Generator(np.random.PCG64(78))
        wu = di.Tensor(g.standard_normal((wl.Hkv, wl.dd, wl.d), dtype=np.float32) /
                       np.sqrt(wl.dd), wl.dtype)
    cap = L0 + steps
    c = dar.DarCache(wl.B, wl.Hkv, wl.d, wl.dd, wl.w, cap, TDT[wl.dtype])
    wdd, wud = to_dev(wd), to_dev(wu)
    if L0 > 0:
        dar.dar_cache_append(c, to_dev(pre["k"]), to_dev(pre["v"]), wdd, Hq=wl.Hq)
    rope = dar.Rope(r, base, n_pos=cap)
    grp = wl.Hq // wl.Hkv
    heads = check_heads or [(b, h) for b in range(wl.B) for h in range(wl.Hq)]
    hist_k, hist_v = {}, {}
    for (b, h) in heads:
        key = (b, h // grp)
        if key not in hist_k:
            hist_k[key] = [pre["k"].f64_slice(key)]
            hist_v[key] = [pre["v"].f64_slice(key)]
    worst = 0.0
    for t in range(steps):
        st = di.make_decode_step(wl, t)
        dar.dar_cache_append(c, to_dev(st["k"]), to_dev(st["v"]), wdd, Hq=wl.Hq)
        o = dar.dar_attn_decode_rope(c, to_dev(st["q"]), wdd, rope, w_up=wud)
        torch.cuda.synchronize()
        got = to_host64(o)
        assert np.isfinite(got).all()
        L = L0 + t + 1
        for key in hist_k:
            hist_k[key].append(st["k"].f64[key[0], key[1]])
            hist_v[key].append(st["v"].f64[key[0], key[1]])
        for (b, h) in heads:
            g = h // grp
            K = np.concatenate(hist_k[(b, g)])
            V = np.concatenate(hist_v[(b, g)])
            ref = oracle.rows_rope(K, V, wd.f64[g], None if wu is None else wu.f64[g], wl.w, r,
                                   base, 0, [L - 1], st["q"].f64[b, h][None])
            worst = max(worst, float(np.abs(got[b, h] - ref[0]).max()))
    assert worst <= tol(wl.dtype), worst
    return worst


DEC = di.Workload("dec_rope", 33, 2, 8, 2, 0, 64, 16, 32, "bf16", kind="decode")


@pytest.mark.parametrize("w", [0, 1, 32, 600])
@pytest.mark.parametrize("r", [64, 16])
def test_decode_rope_bf16(w, r):
    run_decode_rope(DEC.with_(w=w), 300, 2, r, untied=(w == 1))


def test_decode_rope_fp32_tiny():
    run_decode_rope(di.Workload("dec_rope_tiny", 34, 1, 2, 2, 0, 16, 4, 8, "f32", kind="decode"),
                    50, 3, 16)


@pytest.mark.parametrize("G", [1, 2, 8])
def test_decode_rope_group_sizes(G):
    run_decode_rope(DEC.with_(Hq=2 * G, Hkv=2), 130, 2, 32, base=500000.0)


def test_decode_rope_d128_long():
    run_decode_rope(di.Workload("dec_rope_d128", 35, 1, 8, 2, 0, 128, 32, 100, "bf16",
                                kind="decode"), 3000, 2, 128, base=500000.0)


@pytest.mark.parametrize("dd,r,w,L0,untied", [
    (32, 32, 64, 700, False), (16, 64, 100, 300, True), (32, 16, 0, 400, False),
    (32, 64, 512, 600, True),
    # few (batch, KV head) pairs and long caches: split records and the combine
    (32, 32, 256, 20000, False), (16, 16, 1024, 9000, True),
])
def test_decode_rope_d128_matrix_core(dd, r, w, L0, untied):
    """d = 128 on the matrix cores: the first 64 elements of each distant key
    lifted and rotated, the unrotated upper half absorbed in the query."""
    run_decode_rope(DEC.with_(B=1, d=128, dd=dd, w=w), L0, 2, r, untied=untied)


def test_decode_rope_starts_from_empty_cache():
    run_decode_rope(DEC.with_(w=4), 0, 7, 64)


def test_decode_rope_matches_prefill_rope_rows():
    """Decoding token p after appending tokens 0..p gives row p of the
    prefill with the same rotary embedding."""
    wl = di.Workload("dec_vs_prefill_rope", 36, 1, 4, 2, 160, 64, 16, 24, "bf16")
    inp = di.make_prefill_inputs(wl)
    q, k, v, wd = (to_dev(inp[x]) for x in ("q", "k", "v", "wd"))
    rope = dar.Rope(64, 10000.0, n_pos=wl.T)
    o_pre = dar.dar_attn_prefill_rope(q, k, v, wd, None, wl.w, rope)
    c = dar.DarCache(wl.B, wl.Hkv, wl.d, wl.dd, wl.w, wl.T, torch.bfloat16)
    worst = 0.0
    for p in range(wl.T):
        dar.dar_cache_append(c, k[:, :, p:p + 1].contiguous(), v[:, :, p:p + 1].contiguous(), wd,
                             Hq=wl.Hq)
        if p % 13 == 0 or p in (wl.w - 1, wl.w, wl.T - 1):
            o = dar.dar_attn_decode_rope(c, q[:, :, p].contiguous(), wd, rope)
            worst = max(worst, (o.float() - o_pre[:, :, p].float()).abs().max().item())
    torch.cuda.synchronize()
    assert worst <= 2e-2, worst


def test_decode_rope_full_size_sampled_heads():
    """The decode1b cache (B32 Hq32 Hkv8 d64 d_down16 w512, 32768 tokens) with
    full rotation: sampled heads against the oracle."""
    wl = di.WORKLOADS["decode1b"]
    run_decode_rope(wl, wl.T, 1, 64, check_heads=[(0, 0), (5, 9), (31, 31)])


@pytest.mark.parametrize("L0,dd,r,untied", [(20000, 16, 64, False), (9000, 32, 32, True),
                                            (5000, 32, 16, False), (700, 32, 64, True)])
def test_decode_rope_matrix_core_shapes(L0, dd, r, untied):
    """d_down 32 and long caches over few (batch, KV head) pairs: each pair is
    split over several workgroups whose partial records the combine kernel
    merges."""
    run_decode_rope(DEC.with_(B=1, dd=dd, w=256), L0, 2, r, base=500000.0, untied=untied)
