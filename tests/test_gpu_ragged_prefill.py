"""GPU parity of the ragged-batch prefill (dar_attn_prefill_ragged through the
C ABI): sequence b of a padded batch holds seq_lens[b] tokens. Every row
i < seq_lens[b] is compared with the fp64 oracle's prefill over that
sequence's own positions 0..seq_lens[b]-1 (Eq. 3-4); the padding positions of
q, k and v hold NaN, so a kernel that read one would show it, and the rows of
o and lse past each length must keep what the caller put there.
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

SENTINEL = 7.0


def run_ragged(wl, lens, untied=False, check_lse=True, rows_only=None):
    inp = di.make_prefill_inputs(wl, untied=untied)
    T = wl.T
    q, k, v = to_dev(inp["q"]), to_dev(inp["k"]), to_dev(inp["v"])
    for b, L in enumerate(lens):
        for x in (q, k, v):
            x[b, :, L:] = float("nan")
    wd, wu = to_dev(inp["wd"]), to_dev(inp["wu"])
    sl = torch.tensor(lens, dtype=torch.int32, device=q.device)
    o = torch.full_like(q, SENTINEL)
    lse = torch.full((wl.B, wl.Hq, T), SENTINEL, dtype=torch.float32, device=q.device)
    dar.dar_attn_prefill_ragged(q, k, v, wd, wu, wl.w, sl, o=o, lse=lse, return_lse=True)
    torch.cuda.synchronize()
    got = to_host64(o)
    got_lse = lse.double().cpu().numpy()
    worst = 0.0
    for b, L in enumerate(lens):
        assert (got[b, :, L:] == SENTINEL).all(), "row past the length written (b=%d)" % b
        assert (got_lse[b, :, L:] == SENTINEL).all()
        if L == 0:
            continue
        sub = lambda t: t.f64[b:b + 1, :, :L]
        if rows_only is None:
            ref, ref_lse = oracle.prefill(sub(inp["q"]), sub(inp["k"]), sub(inp["v"]), inp["wd"].f64,
                                          None if inp["wu"] is None else inp["wu"].f64, wl.w,
                                          want_lse=True)
            g = got[b:b + 1, :, :L]
            assert np.isfinite(g).all()
            worst = max(worst, float(np.abs(g - ref).max()))
            if check_lse:
                assert np.abs(got_lse[b:b + 1, :, :L] - ref_lse).max() <= (
                    1e-4 if wl.dtype == "f32" else 2e-2)
        else:
            grp = wl.Hq // wl.Hkv
            rows = np.array(sorted({r for r in rows_only(L)}))
            for h in (0, wl.Hq - 1):
                gg = h // grp
                ref = oracle.rows(inp["k"].f64[b, gg, :L], inp["v"].f64[b, gg, :L], inp["wd"].f64[gg],
                                  None, wl.w, rows, inp["q"].f64[b, h, rows])
                worst = max(worst, float(np.abs(got[b, h, rows] - ref).max()))
    assert worst <= tol(wl.dtype), worst
    return worst


BF16 = di.Workload("ragged_bf16", 45, 6, 4, 2, 300, 64, 16, 64, "bf16")
LENS = [300, 1, 0, 37, 257, 129]


@pytest.mark.parametrize("w", [0, 1, 32, 64, 100, 299, 400])
def test_bf16_matrix_core_windows(w):
    run_ragged(BF16.with_(w=w), LENS)


@pytest.mark.parametrize("d,dd,G", [(64, 32, 2), (128, 32, 4), (128, 16, 1), (64, 16, 8)])
def test_bf16_matrix_core_shapes(d, dd, G):
    run_ragged(BF16.with_(d=d, dd=dd, Hq=2 * G, Hkv=2, w=48), LENS, untied=(d == 128))


def test_fp32_generic():
    wl = di.WORKLOADS["tiny"].with_(B=4, Hq=4, Hkv=2, T=90, w=16)
    run_ragged(wl, [90, 5, 0, 61])


def test_bf16_generic_shape():
    run_ragged(di.Workload("ragged_generic", 46, 3, 4, 2, 150, 80, 20, 30, "bf16"), [150, 77, 2])


def test_all_full_equals_dense():
    """seq_lens all T: the same bits as dar_attn_prefill."""
    wl = BF16.with_(w=64, B=2)
    inp = di.make_prefill_inputs(wl)
    q, k, v, wd = (to_dev(inp[x]) for x in ("q", "k", "v", "wd"))
    o1 = dar.dar_attn_prefill(q, k, v, wd, None, wl.w)
    sl = torch.full((wl.B,), wl.T, dtype=torch.int32, device=q.device)
    o2 = dar.dar_attn_prefill_ragged(q, k, v, wd, None, wl.w, sl)
    torch.cuda.synchronize()
    assert torch.equal(o1.view(torch.int16), o2.view(torch.int16))


def test_full_size_ragged_pythia70m():
    """pythia70m shape (B8 H8 T2048 d64 d_down16 w256) with lengths 1..2048:
    every row of every head of every sequence."""
    wl = di.WORKLOADS["pythia70m"]
    lens = [2048, 1, 255, 256, 257, 1000, 1777, 2047]
    run_ragged(wl, lens)
