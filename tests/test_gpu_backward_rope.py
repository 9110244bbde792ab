"""GPU backward of the prefill with the rotary embedding of Eq. 3
(dar_attn_prefill_rope_backward through the C ABI) against the fp64 oracle's
rotary backward on the same seeded inputs.

The GPU backward is fed the GPU rotary forward's own o and lse. Tolerance as
for the plain backward: the forward's bf16 bound 2e-2 relative to each
gradient tensor's scale,
  max |got - ref| <= tol * max(1, max |ref|)   per tensor (dq, dk, dv, dW),
and an elementwise bound |got - ref| <= B * tol * max(1, |ref|) with B from
ELEM_BOUND (the gradients are sums with cancellation: an element's error
follows the terms that built it, and the weight gradients sum over every row
of the batch).
"""
import numpy as np
import pytest
import torch

import dar_inputs as di
from oracle import oracle
from tests.dev import to_dev, to_host64, tol

pytestmark = pytest.mark.gpu

dar = pytest.importorskip("paper_2606_18587_amd")

ELEM_BOUND = {"dq": 1.4, "dk": 1.4, "dv": 1.4, "dwd": 12.0, "dwu": 12.0}


def compare(got, ref, what):
    t = tol("bf16")
    worst = {}
    for n, a, b in zip(("dq", "dk", "dv", "dwd", "dwu"), got, ref):
        if b is None:
            assert a is None, n
            continue
        assert a.shape == b.shape, (n, a.shape, b.shape)
        assert np.isfinite(a).all(), what + " " + n + " not finite"
        err = np.abs(a - b)
        ratio = err.max() / (t * max(1.0, np.abs(b).max()))
        elem = (err / (t * np.maximum(1.0, np.abs(b)))).max()
        worst[n] = ratio
        worst[n + "_elem"] = elem
        assert ratio <= 1.0, "%s %s: error %.3g of the normwise bound (max abs err %.3g)" % (
            what, n, ratio, err.max())
        assert elem <= ELEM_BOUND[n], "%s %s: elementwise error %.3g of the bound" % (what, n, elem)
    return worst


def run_gpu(inp, w, r, base, pos0):
    q, k, v = to_dev(inp["q"]), to_dev(inp["k"]), to_dev(inp["v"])
    wd, wu = to_dev(inp["wd"]), to_dev(inp["wu"])
    dout = to_dev(inp["dout"])
    T = q.shape[2]
    rope = dar.Rope(r, base, n_pos=pos0 + T)
    o, lse = dar.dar_attn_prefill_rope(q, k, v, wd, wu, w, rope, pos0=pos0, return_lse=True)
    grads = dar.dar_attn_prefill_rope_backward(q, k, v, wd, wu, w, rope, o, lse, dout, pos0=pos0)
    torch.cuda.synchronize()
    return [None if g is None else to_host64(g) for g in grads]


def full_compare(wl, r, untied=False, base=10000.0, pos0=0, seed_shift=0):
    inp = di.make_backward_inputs(wl, untied=untied, seed_shift=seed_shift)
    got = run_gpu(inp, wl.w, r, base, pos0)
    ref = oracle.backward_rope(inp["q"].f64, inp["k"].f64, inp["v"].f64, inp["wd"].f64,
                               None if inp["wu"] is None else inp["wu"].f64, wl.w, r, base,
                               inp["dout"].f64, pos0=pos0)
    worst = compare(got, ref, "%s w=%d T=%d r=%d" % (wl.name, wl.w, wl.T, r))
    print(wl.name, wl.w, wl.T, r, " ".join("%s=%.3f" % kv for kv in worst.items()))
    return worst


BF16_SMALL = di.Workload("rope_bwd_small", 50, 1, 4, 2, 300, 64, 16, 128, "bf16")


@pytest.mark.parametrize("w", [0, 1, 64, 128, 299, 300, 1000])
@pytest.mark.parametrize("untied", [False, True])
def test_d64_window_sweep(w, untied):
    full_compare(BF16_SMALL.with_(w=w), 16 if w % 2 == 0 else 64, untied=untied)


@pytest.mark.parametrize("T", [1, 2, 61, 129, 257])
def test_d64_ragged_lengths(T):
    full_compare(BF16_SMALL.with_(T=T, w=32, B=2), 32)


@pytest.mark.parametrize("w,r,untied", [(0, 128, False), (100, 32, True), (512, 64, False)])
def test_d128_gqa(w, r, untied):
    full_compare(di.Workload("rope_bwd_d128", 51, 1, 8, 2, 400, 128, 32, w, "bf16"), r,
                 untied=untied, base=500000.0)


@pytest.mark.parametrize("d,dd,w,T,r", [(64, 32, 40, 333, 64), (128, 16, 77, 290, 16),
                                        (64, 8, 33, 97, 24), (128, 48, 50, 150, 2)])
def test_other_shapes_and_rotary_dims(d, dd, w, T, r):
    """d_down 8 and 48, rotary dims that are not multiples of 16."""
    full_compare(di.Workload("rope_bwd_mixed", 52, 2, 4, 1, T, d, dd, w, "bf16"), r, untied=True)


def test_offset_positions_and_zero_rotary_dim():
    """Rows at positions 77.. of a longer sequence, and r = 0, whose gradients
    are those of the plain backward (checked against the oracle's)."""
    wl = BF16_SMALL.with_(w=48, T=200)
    full_compare(wl, 64, pos0=77, base=500000.0)
    inp = di.make_backward_inputs(wl, untied=True, seed_shift=3)
    got = run_gpu(inp, wl.w, 0, 10000.0, 0)
    ref = oracle.backward(inp["q"].f64, inp["k"].f64, inp["v"].f64, inp["wd"].f64,
                          inp["wu"].f64, wl.w, inp["dout"].f64)
    compare(got, ref, "r=0 against the plain backward")


def test_deterministic():
    wl = BF16_SMALL.with_(w=64, T=333, B=2)
    inp = di.make_backward_inputs(wl, untied=True)
    a = run_gpu(inp, wl.w, 32, 10000.0, 5)
    b = run_gpu(inp, wl.w, 32, 10000.0, 5)
    for x, y in zip(a, b):
        assert (x is None and y is None) or np.array_equal(x, y)


def test_full_size_pythia70m_one_head():
    """B8 H8 T2048 d64 d_down16 w256 with rotary dimension 16 (the Pythia
    models' rotary width) on the GPU; the oracle recomputes the gradients of
    one KV head over the whole batch (dq/dk/dv of its rows and the head's full
    dW_down)."""
    wl = di.WORKLOADS["pythia70m"]
    inp = di.make_backward_inputs(wl)
    got = run_gpu(inp, wl.w, 16, 10000.0, 0)
    g = 2
    G = wl.Hq // wl.Hkv
    hs = slice(g * G, (g + 1) * G)
    ref = oracle.backward_rope(inp["q"].f64[:, hs], inp["k"].f64[:, g:g + 1], inp["v"].f64[:, g:g + 1],
                               inp["wd"].f64[g:g + 1], None, wl.w, 16, 10000.0, inp["dout"].f64[:, hs])
    sub = [got[0][:, hs], got[1][:, g:g + 1], got[2][:, g:g + 1], got[3][g:g + 1], None]
    worst = compare(sub, ref, "pythia70m rope head %d" % g)
    print("pythia70m rope head", g, " ".join("%s=%.3f" % kv for kv in worst.items()))
