"""The prefill and the decode captured into a HIP graph (through torch's graph
capture on the current stream) and replayed: every replay, with eager work
and synchronisations in between, must give the eager call's bits. Nothing in
these entry points allocates, memsets or synchronises, so they can be
captured."""
import numpy as np
import pytest
import torch

import dar_inputs as di
from tests.dev import to_dev

pytestmark = pytest.mark.gpu

dar = pytest.importorskip("paper_2606_18587_amd")


def bits(x):
    return x.detach().cpu().view(torch.int16).numpy().copy()


def replay_matches(run, out):
    """Capture run() (which writes `out`), replay it three times with eager
    work between the replays; each replay must reproduce the eager bits."""
    run()
    torch.cuda.synchronize()
    ref = bits(out)
    g = torch.cuda.CUDAGraph()
    cs = torch.cuda.Stream()
    cs.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(cs):
        with torch.cuda.graph(g, stream=cs):
            run()
    torch.cuda.current_stream().wait_stream(cs)
    torch.cuda.synchronize()
    scratch = torch.zeros(1 << 20, device="cuda")
    for rep in range(3):
        out.fill_(float("nan"))        # eager work between replays
        scratch.add_(1.0)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert np.array_equal(bits(out), ref), "replay %d differs" % rep


@pytest.mark.parametrize("w", [0, 64])
def test_prefill_graph_replay(w):
    wl = di.Workload("graph_pf", 70, 2, 4, 2, 700, 64, 16, w, "bf16")
    inp = di.make_prefill_inputs(wl)
    q, k, v, wd = (to_dev(inp[x]) for x in ("q", "k", "v", "wd"))
    o = torch.empty_like(q)
    shape = dar.make_shape(wl.B, wl.Hq, wl.Hkv, wl.d, wl.dd, wl.w, torch.bfloat16)
    ws = torch.empty(dar.dar_prefill_workspace_bytes(shape, wl.T), dtype=torch.uint8, device="cuda")
    replay_matches(lambda: dar.dar_attn_prefill(q, k, v, wd, None, wl.w, o=o, ws=ws), o)


@pytest.mark.parametrize("L0", [300, 20000])
def test_decode_graph_replay(L0):
    """Decode over a fixed cache (one workgroup per (batch, KV head) at the
    short length; split records and the combine kernel at the long one)."""
    wl = di.Workload("graph_dec", 71, 1, 8, 2, 0, 64, 16, 32, "bf16", kind="decode")
    pre = di.make_decode_prefix(wl, L0)
    c = dar.DarCache(wl.B, wl.Hkv, wl.d, wl.dd, wl.w, L0, torch.bfloat16)
    wd = to_dev(pre["wd"])
    dar.dar_cache_append(c, to_dev(pre["k"]), to_dev(pre["v"]), wd, Hq=wl.Hq)
    q = to_dev(di.make_decode_step(wl, 0)["q"])
    o = torch.empty_like(q)
    shape = dar.make_shape(wl.B, wl.Hq, wl.Hkv, wl.d, wl.dd, wl.w, torch.bfloat16)
    ws = torch.empty(dar.dar_decode_workspace_bytes(shape, c.cap), dtype=torch.uint8, device="cuda")
    replay_matches(lambda: dar.dar_attn_decode(c, q, wd, o=o, ws=ws), o)
    replay_matches(lambda: dar.dar_attn_decode_noalloc(c, q, wd, o=o), o)


def test_paged_decode_graph_replay():
    """Paged decode, plain and with the rotary embedding, over a batch of
    mixed lengths: a long sequence split into parts (their records merged by
    the combine kernel, which reads the record counts the decode kernel
    wrote), short ones finished whole, an empty one written as NaN."""
    B, Hq, Hkv, d, dd, w, ps = 6, 8, 2, 64, 16, 32, 64
    lens = [9000, 5, 0, 300, 64, 1]
    nblk = max(lens) // ps + 2
    n_pages = B * nblk
    pc = dar.DarPagedCache(B, Hkv, d, dd, w, ps, nblk, n_pages, torch.bfloat16)
    gen = torch.Generator(device="cuda").manual_seed(73)
    for t in (pc.k_win, pc.v_win, pc.k_pool, pc.v_pool):
        t.copy_(torch.randn(t.shape, device="cuda", generator=gen))
    perm = torch.randperm(n_pages, generator=torch.Generator().manual_seed(74))
    pc.block_table.copy_(perm.view(B, nblk).to(torch.int32))
    pc.lens.copy_(torch.tensor(lens, dtype=torch.int32))
    q = torch.randn(B, Hq, d, device="cuda", generator=gen).bfloat16()
    wd = (torch.randn(Hkv, d, dd, device="cuda", generator=gen) / d ** 0.5).bfloat16()
    o = torch.empty_like(q)
    shape = dar.make_shape(B, Hq, Hkv, d, dd, w, torch.bfloat16)
    ws = torch.empty(dar.dar_decode_workspace_bytes(shape, pc.cap), dtype=torch.uint8, device="cuda")
    replay_matches(lambda: dar.dar_attn_decode_paged(pc, q, wd, o=o, ws=ws), o)
    got = o.float().cpu()
    assert torch.isnan(got[2]).all() and torch.isfinite(got[[0, 1, 3, 4, 5]]).all()
    # the rotary form over the same batch (its table filled before the capture)
    rope = dar.Rope(64, 10000.0, n_pos=pc.cap)
    replay_matches(lambda: dar.dar_attn_decode_paged_rope(pc, q, wd, rope, o=o, ws=ws), o)
    got = o.float().cpu()
    assert torch.isnan(got[2]).all() and torch.isfinite(got[[0, 1, 3, 4, 5]]).all()
