"""GPU prefill parity: dar_attn_prefill (through the C ABI) against the fp64
oracle on the same seeded inputs, element by element.

Tolerance (max abs, unit-scale data): 1e-4 for fp32, 2e-2 for bf16 storage
with fp32 accumulation.
"""
import numpy as np
import pytest
import torch

import dar_inputs as di
from oracle import oracle
from tests.dev import to_dev, to_host64, tol

pytestmark = pytest.mark.gpu

dar = pytest.importorskip("paper_2606_18587_amd")


def run_gpu(inp, w, want_lse=False):
    """dar_attn_prefill (or dar_attn_prefill_lse) into NaN-filled outputs, so a
    row the kernels never write cannot pass as a stale value."""
    q, k, v = to_dev(inp["q"]), to_dev(inp["k"]), to_dev(inp["v"])
    wd, wu = to_dev(inp["wd"]), to_dev(inp["wu"])
    o = torch.full_like(q, float("nan"))
    if want_lse:
        lse = torch.full(q.shape[:3], float("nan"), dtype=torch.float32, device=q.device)
        dar.dar_attn_prefill_lse(q, k, v, wd, wu, w, o=o, lse=lse)
        torch.cuda.synchronize()
        return o, lse
    dar.dar_attn_prefill(q, k, v, wd, wu, w, o=o)
    torch.cuda.synchronize()
    return o


def full_compare(wl, untied=False, seed_shift=0, q_scale=1.0):
    inp = di.make_prefill_inputs(wl, untied=untied, seed_shift=seed_shift, q_scale=q_scale)
    o = to_host64(run_gpu(inp, wl.w))
    ref = oracle.prefill(inp["q"].f64, inp["k"].f64, inp["v"].f64, inp["wd"].f64,
                         None if inp["wu"] is None else inp["wu"].f64, wl.w)
    err = np.abs(o - ref)
    assert np.isfinite(o).all()
    assert err.max() <= tol(wl.dtype), "max abs err %.3g at %s" % (
        err.max(), np.unravel_index(err.argmax(), err.shape))
    return err.max()


def test_tiny_fp32_workload():
    full_compare(di.WORKLOADS["tiny"])


@pytest.mark.parametrize("w", [0, 1, 8, 63, 64, 65, 200])
def test_tiny_fp32_window_sweep(w):
    full_compare(di.WORKLOADS["tiny"].with_(w=w, T=100, B=2, Hq=4, Hkv=2), untied=(w % 2 == 1))


BF16_SMALL = di.Workload("bf16_small", 10, 1, 4, 2, 300, 64, 16, 128, "bf16")


@pytest.mark.parametrize("w", [0, 1, 16, 64, 128, 129, 299, 300, 1000])
@pytest.mark.parametrize("untied", [False, True])
def test_bf16_d64_window_sweep(w, untied):
    full_compare(BF16_SMALL.with_(w=w), untied=untied)


@pytest.mark.parametrize("T", [1, 2, 61, 127, 128, 129, 257, 500])
def test_bf16_d64_ragged_lengths(T):
    full_compare(BF16_SMALL.with_(T=T, w=32, B=2))


@pytest.mark.parametrize("w", [0, 64, 100, 512])
def test_bf16_d128_gqa(w):
    full_compare(di.Workload("bf16_d128", 11, 1, 8, 2, 400, 128, 32, w, "bf16"), untied=(w == 100))


@pytest.mark.parametrize("d,dd,w,T", [(64, 32, 40, 333), (128, 16, 77, 290), (64, 16, 33, 97)])
@pytest.mark.parametrize("untied", [False, True])
def test_bf16_other_matrix_core_shapes(d, dd, w, T, untied):
    full_compare(di.Workload("bf16_mixed", 13, 2, 4, 1, T, d, dd, w, "bf16"), untied=untied)


def test_bf16_peaky_queries():
    # queries scaled by 4: sharp softmax rows, large running-max changes
    full_compare(BF16_SMALL.with_(w=64, T=400), q_scale=4.0)


@pytest.mark.parametrize("shape", [(1, 3, 1, 90, 48, 12, 10), (2, 2, 2, 70, 32, 32, 5),
                                   (1, 2, 1, 50, 256, 64, 7)])
def test_generic_shapes(shape):
    B, Hq, Hkv, T, d, dd, w = shape
    for dt in ("f32", "bf16"):
        full_compare(di.Workload("generic", 12, B, Hq, Hkv, T, d, dd, w, dt), untied=True)


def test_deterministic():
    inp = di.make_prefill_inputs(BF16_SMALL)
    a = run_gpu(inp, BF16_SMALL.w)
    b = run_gpu(inp, BF16_SMALL.w)
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))


def test_gqa_equals_repeated_mha():
    wl = BF16_SMALL.with_(Hq=4, Hkv=2, T=200, w=50)
    inp = di.make_prefill_inputs(wl, untied=True)
    q, k, v = to_dev(inp["q"]), to_dev(inp["k"]), to_dev(inp["v"])
    wd, wu = to_dev(inp["wd"]), to_dev(inp["wu"])
    o1 = dar.dar_attn_prefill(q, k, v, wd, wu, wl.w)
    rep = lambda x: x.repeat_interleave(2, dim=0 if x.dim() == 3 else 1).contiguous()
    o2 = dar.dar_attn_prefill(q, rep(k), rep(v), rep(wd), rep(wu), wl.w)
    torch.cuda.synchronize()
    assert (o1.float() - o2.float()).abs().max().item() <= 2e-2


# ---------------------------------------------------------------- full sizes

@pytest.mark.parametrize("name", ["pythia70m", "pythia410m_w128", "pythia410m_w512", "long16k"])
def test_full_size_every_row(name):
    """The benchmark prefill workloads at their full size: every row of every
    head, and every row's log-sum-exp, against the oracle (Eq. 3-4). The
    outputs start as NaN, so a row no kernel writes fails."""
    wl = di.WORKLOADS[name]
    inp = di.make_prefill_inputs(wl)
    o, lse = run_gpu(inp, wl.w, want_lse=True)
    got = to_host64(o)
    got_lse = lse.cpu().numpy().astype(np.float64)
    del o, lse
    ref, ref_lse = oracle.prefill(inp["q"].f64, inp["k"].f64, inp["v"].f64, inp["wd"].f64, None,
                                  wl.w, want_lse=True)
    assert np.isfinite(got).all() and np.isfinite(got_lse).all()
    err = np.abs(got - ref)
    lerr = np.abs(got_lse - ref_lse)
    print("[%s] every row: max abs err %.4g (at %s), lse %.4g" % (
        name, err.max(), np.unravel_index(err.argmax(), err.shape), lerr.max()), flush=True)
    assert err.max() <= tol(wl.dtype)
    assert lerr.max() <= tol(wl.dtype)


@pytest.mark.parametrize("wl,untied", [
    (di.WORKLOADS["tiny"], False),
    (di.WORKLOADS["tiny"].with_(w=0, T=100), True),
    (BF16_SMALL.with_(w=64), False),
    (BF16_SMALL.with_(w=0), True),
    (BF16_SMALL.with_(w=1000), False),
    (di.Workload("bf16_d128", 11, 1, 8, 2, 400, 128, 32, 100, "bf16"), True),
    (di.Workload("generic", 14, 1, 2, 1, 50, 256, 64, 7, "bf16"), False),
])
def test_log_sum_exp_output(wl, untied):
    """The optional lse output (log of each row's softmax denominator) against
    the oracle's, max abs error within the path's tolerance."""
    inp = di.make_prefill_inputs(wl, untied=untied)
    q, k, v = to_dev(inp["q"]), to_dev(inp["k"]), to_dev(inp["v"])
    wd, wu = to_dev(inp["wd"]), to_dev(inp["wu"])
    o, lse = dar.dar_attn_prefill(q, k, v, wd, wu, wl.w, return_lse=True)
    o2 = dar.dar_attn_prefill(q, k, v, wd, wu, wl.w)
    torch.cuda.synchronize()
    assert torch.equal(o, o2)  # asking for lse changes nothing else
    ref_o, ref_lse = oracle.prefill(inp["q"].f64, inp["k"].f64, inp["v"].f64, inp["wd"].f64,
                                    None if inp["wu"] is None else inp["wu"].f64, wl.w,
                                    want_lse=True)
    err = np.abs(lse.cpu().numpy().astype(np.float64) - ref_lse)
    assert err.max() <= tol(wl.dtype), "lse max abs err %.3g" % err.max()
