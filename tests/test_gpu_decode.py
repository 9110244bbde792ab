"""GPU decode parity: dar_cache_append + dar_attn_decode (through the C ABI)
against the oracle's row at position len-1 over the full-dimension history."""
import numpy as np
import pytest
import torch

import dar_inputs as di
from oracle import oracle
from tests.dev import to_dev, to_host64, tol

pytestmark = pytest.mark.gpu

dar = pytest.importorskip("paper_2606_18587_amd")

TDT = {"bf16": torch.bfloat16, "f32": torch.float32}


def run_decode(wl, L0, steps, cap=None, untied=False, check_heads=None, check_steps=None):
    """Append a prefix of L0 tokens, then `steps` x {append one, decode}; compare
    the decodes of `check_steps` (default: every step) with the oracle for the
    heads `check_heads` (default: all). The output is NaN-filled before each
    decode, so a head no kernel writes fails. Returns the worst max-abs error."""
    pre = di.make_decode_prefix(wl, L0)
    wd = pre["wd"]
    wu = None
    if untied:
        g = np.random.Generator(np.random.PCG64(77))
        wu = di.Tensor(g.standard_normal((wl.Hkv, wl.dd, wl.d), dtype=np.float32) /
                       np.sqrt(wl.dd), wl.dtype)
    cap = cap or (L0 + steps)
    c = dar.DarCache(wl.B, wl.Hkv, wl.d, wl.dd, wl.w, cap, TDT[wl.dtype])
    wdd, wud = to_dev(wd), to_dev(wu)
    if L0 > 0:
        dar.dar_cache_append(c, to_dev(pre["k"]), to_dev(pre["v"]), wdd, Hq=wl.Hq)
    grp = wl.Hq // wl.Hkv
    heads = check_heads or [(b, h) for b in range(wl.B) for h in range(wl.Hq)]
    # query heads to check, grouped by the (batch, KV head) whose history they read
    groups = {}
    for (b, h) in heads:
        groups.setdefault((b, h // grp), []).append(h)
    check_steps = set(range(steps)) if check_steps is None else set(check_steps)
    new_k, new_v = [], []   # each step's token, kept in storage form
    worst = 0.0
    o = torch.empty(wl.B, wl.Hq, wl.d, dtype=TDT[wl.dtype], device="cuda")
    for t in range(steps):
        st = di.make_decode_step(wl, t)
        new_k.append(st["k"].store)
        new_v.append(st["v"].store)
        dar.dar_cache_append(c, to_dev(st["k"]), to_dev(st["v"]), wdd, Hq=wl.Hq)
        assert c.len == L0 + t + 1
        if t not in check_steps:
            continue
        o.fill_(float("nan"))
        dar.dar_attn_decode(c, to_dev(st["q"]), wdd, wud, o=o)
        torch.cuda.synchronize()
        got = to_host64(o)
        assert np.isfinite(got).all()
        L = L0 + t + 1
        nk = di.Tensor.from_store(np.concatenate(new_k, axis=2), wl.dtype)
        nv = di.Tensor.from_store(np.concatenate(new_v, axis=2), wl.dtype)
        for (b, g), hs in sorted(groups.items()):
            K = np.concatenate([pre["k"].f64_slice((b, g)), nk.f64_slice((b, g))])
            V = np.concatenate([pre["v"].f64_slice((b, g)), nv.f64_slice((b, g))])
            ref = oracle.rows(K, V, wd.f64[g], None if wu is None else wu.f64[g], wl.w,
                              [L - 1] * len(hs), st["q"].f64[b, hs])
            worst = max(worst, float(np.abs(got[b, hs] - ref).max()))
    assert worst <= tol(wl.dtype), worst
    return worst


SMALL = di.Workload("dec_small", 20, 2, 8, 2, 0, 64, 16, 32, "bf16", kind="decode")


def test_decode_small_gqa():
    run_decode(SMALL, 300, 4)


def test_decode_untied():
    run_decode(SMALL, 200, 2, untied=True)


@pytest.mark.parametrize("w", [0, 1, 600])
def test_decode_window_extremes(w):
    run_decode(SMALL.with_(w=w), 150, 3)


def test_decode_starts_from_empty_cache():
    run_decode(SMALL.with_(w=4), 0, 9)


@pytest.mark.parametrize("G", [1, 2, 8])
def test_decode_group_sizes(G):
    run_decode(SMALL.with_(Hq=2 * G, Hkv=2), 130, 2)


def test_decode_fp32_tiny():
    run_decode(di.Workload("dec_tiny", 21, 1, 2, 2, 0, 16, 4, 8, "f32", kind="decode"), 50, 3)


def test_decode_d128():
    run_decode(di.Workload("dec_d128", 22, 1, 8, 2, 0, 128, 32, 100, "bf16", kind="decode"),
               700, 2)


def test_decode_matches_prefill_rows():
    """Decoding token p after appending tokens 0..p gives prefill row p."""
    wl = di.Workload("dec_vs_prefill", 23, 1, 4, 2, 160, 64, 16, 24, "bf16")
    inp = di.make_prefill_inputs(wl)
    q, k, v, wd = (to_dev(inp[x]) for x in ("q", "k", "v", "wd"))
    o_pre = dar.dar_attn_prefill(q, k, v, wd, None, wl.w)
    c = dar.DarCache(wl.B, wl.Hkv, wl.d, wl.dd, wl.w, wl.T, torch.bfloat16)
    worst = 0.0
    for p in range(wl.T):
        dar.dar_cache_append(c, k[:, :, p:p + 1].contiguous(), v[:, :, p:p + 1].contiguous(), wd,
                             Hq=wl.Hq)
        if p % 13 == 0 or p in (wl.w - 1, wl.w, wl.T - 1):
            o = dar.dar_attn_decode(c, q[:, :, p].contiguous(), wd)
            worst = max(worst, (o.float() - o_pre[:, :, p].float()).abs().max().item())
    torch.cuda.synchronize()
    assert worst <= 2e-2, worst


def test_decode_full_size_128_steps():
    """The 1B-scale decode workload as specified: 32768 cached tokens, then
    128 steps of {append, decode}; all 1024 (batch, query head) outputs
    compared with the oracle at steps 1, 64 and 128."""
    wl = di.WORKLOADS["decode1b"]
    worst = run_decode(wl, wl.T, wl.steps, cap=wl.T + wl.steps, check_steps=(0, 63, 127))
    print("[decode1b] 128 steps, every head at steps 1/64/128: max abs err %.4g" % worst,
          flush=True)


@pytest.mark.parametrize("L0,d,dd,untied", [(5000, 64, 16, False), (20000, 64, 16, True),
                                             (3000, 128, 32, False), (9000, 64, 32, False)])
def test_decode_several_workgroups_per_head(L0, d, dd, untied):
    """Few (batch, KV head) pairs and a long cache: each pair is split over
    several workgroups whose partial records the combine kernel merges."""
    run_decode(SMALL.with_(d=d, dd=dd), L0, 2, untied=untied)
