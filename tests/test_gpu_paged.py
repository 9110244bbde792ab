"""GPU parity of the paged split cache with one length per sequence
(dar_cache_append_paged, dar_attn_decode_paged and its rotary variant
dar_attn_decode_paged_rope through the C ABI).

Sequences of different lengths share one batch; their latents live in pages
handed out through a shuffled block table. Each sequence's decode is checked
against the oracle's row at its own position len_b - 1 over its own
full-dimension history (Eq. 3-4, tolerance 2e-2 for bf16), and the pages and
rings written by the paged append are checked byte for byte against a dense
cache that dar_cache_append fills with the same tokens. The rotary decode
is checked against the oracle's rotary row (Eq. 3 with RoPE: query at
position len_b - 1, token e at position e).
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


class Ragged:
    """B sequences with their own prefixes (seeded N(0,1) keys and values),
    each kept in a dense B=1 cache (filled by dar_cache_append) and copied
    into the paged cache: ring rows as they are, latent rows into the pages
    the block table names."""

    def __init__(self, wl, lens, page_size, extra_blocks=1, seed=600, steps=2):
        self.wl, self.ps = wl, page_size
        self.lens = list(lens)
        B = len(lens)
        self.B = B
        g = np.random.Generator(np.random.PCG64(seed))
        self.wd = di.Tensor(g.standard_normal((wl.Hkv, wl.d, wl.dd), dtype=np.float32) /
                            np.sqrt(wl.d), "bf16")
        tot = [L + steps for L in lens]
        self.k = [di.Tensor(g.standard_normal((wl.Hkv, n, wl.d), dtype=np.float32), "bf16") for n in tot]
        self.v = [di.Tensor(g.standard_normal((wl.Hkv, n, wl.d), dtype=np.float32), "bf16") for n in tot]
        self.wdd = to_dev(self.wd)
        maxb = max((n + page_size - 1) // page_size for n in tot) + extra_blocks
        n_pages = sum((n + page_size - 1) // page_size for n in tot) + 3
        self.pc = dar.DarPagedCache(B, wl.Hkv, wl.d, wl.dd, wl.w, page_size, maxb, n_pages,
                                    torch.bfloat16)
        perm = g.permutation(n_pages)
        bt = np.full((B, maxb), -1, np.int32)
        nxt = 0
        for b, n in enumerate(tot):
            for blk in range((n + page_size - 1) // page_size):
                bt[b, blk] = perm[nxt]
                nxt += 1
        self.bt = bt
        self.pc.block_table.copy_(torch.from_numpy(bt))
        self.kdev = [to_dev(x) for x in self.k]
        self.vdev = [to_dev(x) for x in self.v]
        self.dense = []
        for b, L in enumerate(lens):
            c = dar.DarCache(1, wl.Hkv, wl.d, wl.dd, wl.w, L + steps, torch.bfloat16)
            kb = self.kdev[b][None]
            vb = self.vdev[b][None]
            if L > 0:
                dar.dar_cache_append(c, kb[:, :, :L].contiguous(), vb[:, :, :L].contiguous(), self.wdd,
                                     Hq=wl.Hq)
            self.dense.append(c)
            self.scatter(b)
        self.pc.lens.copy_(torch.tensor(lens, dtype=torch.int32))
        torch.cuda.synchronize()

    def scatter(self, b):
        """Copy dense cache b into the paged cache (test-side data movement)."""
        c, L, ps = self.dense[b], self.dense[b].len, self.ps
        if self.wl.w > 0:
            self.pc.k_win[b].copy_(c.k_win[0])
            self.pc.v_win[b].copy_(c.v_win[0])
        for e0 in range(0, max(0, L - self.wl.w), ps):
            e1 = min(e0 + ps, L - self.wl.w)
            page = int(self.bt[b, e0 // ps])
            self.pc.k_pool[page, :, : e1 - e0].copy_(c.k_lat[0, :, e0:e1])
            self.pc.v_pool[page, :, : e1 - e0].copy_(c.v_lat[0, :, e0:e1])

    def step_tokens(self, t):
        """The t-th new token of every sequence: [B,Hkv,d] each."""
        k = torch.stack([self.kdev[b][:, self.lens[b] + t] for b in range(self.B)])
        v = torch.stack([self.vdev[b][:, self.lens[b] + t] for b in range(self.B)])
        return k.contiguous(), v.contiguous()

    def check_decode(self, t, heads_per_seq=None, seed=0, rope=None, wu=None):
        """Decode a fresh query per sequence at its current length; compare
        with the oracle row (with rope: the rotary decode against the
        oracle's rotary row, query at position len - 1, token e at e)."""
        wl = self.wl
        g = np.random.Generator(np.random.PCG64(700 + t + seed))
        q = di.Tensor(g.standard_normal((self.B, wl.Hq, wl.d), dtype=np.float32), "bf16")
        if rope is None:
            o = dar.dar_attn_decode_paged(self.pc, to_dev(q), self.wdd, w_up=to_dev(wu))
        else:
            o = dar.dar_attn_decode_paged_rope(self.pc, to_dev(q), self.wdd, rope, w_up=to_dev(wu))
        torch.cuda.synchronize()
        got = to_host64(o)
        grp = wl.Hq // wl.Hkv
        worst = 0.0
        for b in range(self.B):
            L = self.lens[b] + t
            if L < 1:  # empty sequence: no query position
                assert np.isnan(got[b]).all()
                continue
            assert np.isfinite(got[b]).all()
            heads = range(wl.Hq) if heads_per_seq is None else heads_per_seq
            for h in heads:
                gg = h // grp
                K, V = self.k[b].f64_slice(gg)[:L], self.v[b].f64_slice(gg)[:L]
                wug = None if wu is None else wu.f64[gg]
                if rope is None:
                    ref = oracle.rows(K, V, self.wd.f64[gg], wug, wl.w, [L - 1], q.f64[b, h][None])
                else:
                    ref = oracle.rows_rope(K, V, self.wd.f64[gg], wug, wl.w, rope.rotary_dim,
                                           rope.base, 0, [L - 1], q.f64[b, h][None])
                worst = max(worst, float(np.abs(got[b, h] - ref[0]).max()))
        assert worst <= tol("bf16"), worst
        return worst

    def append_step(self, t):
        """Paged append of token t of every sequence, dense append of the same
        token; the paged cache's new rows must equal the dense cache's."""
        k, v = self.step_tokens(t)
        dar.dar_cache_append_paged(self.pc, k, v, self.wdd, Hq=self.wl.Hq)
        for b in range(self.B):
            dar.dar_cache_append(self.dense[b], k[b:b + 1, :, None].contiguous(),
                                 v[b:b + 1, :, None].contiguous(), self.wdd, Hq=self.wl.Hq)
        torch.cuda.synchronize()
        lens_now = self.pc.lens.cpu().numpy()
        assert lens_now.tolist() == [L + t + 1 for L in self.lens]
        w, ps = self.wl.w, self.ps
        for b in range(self.B):
            L = self.lens[b] + t + 1
            c = self.dense[b]
            if w > 0:
                assert np.array_equal(raw(self.pc.k_win[b]), raw(c.k_win[0]))
                assert np.array_equal(raw(self.pc.v_win[b]), raw(c.v_win[0]))
            ex = L - 1 - w   # the latent this append wrote
            if ex >= 0:
                page = int(self.bt[b, ex // ps])
                assert np.array_equal(raw(self.pc.k_pool[page, :, ex % ps]), raw(c.k_lat[0, :, ex]))
                assert np.array_equal(raw(self.pc.v_pool[page, :, ex % ps]), raw(c.v_lat[0, :, ex]))


WL = di.Workload("paged", 60, 1, 8, 2, 0, 64, 16, 32, "bf16", kind="decode")


@pytest.mark.parametrize("w,ps", [(32, 64), (0, 32), (1, 256), (600, 64)])
def test_ragged_decode_and_append(w, ps):
    r = Ragged(WL.with_(w=w), [1, 37, 300, 64, 511, 129], ps)
    for t in range(2):
        r.check_decode(t)
        r.append_step(t)
    r.check_decode(2)


@pytest.mark.parametrize("d,dd,G", [(64, 32, 4), (128, 16, 2), (128, 32, 8), (64, 16, 1)])
def test_other_shapes(d, dd, G):
    r = Ragged(WL.with_(d=d, dd=dd, Hq=2 * G, Hkv=2, w=48), [5, 200, 97], 64)
    r.check_decode(0)
    r.append_step(0)
    r.check_decode(1)


def test_long_sequences_several_workgroups():
    """Few sequences with long caches: each (sequence, KV head) is split over
    several workgroups (partial records merged by the combine kernel)."""
    r = Ragged(WL.with_(w=256), [20000, 3000], 256, steps=1)
    r.check_decode(0, heads_per_seq=[0, 3, 7])
    r.append_step(0)
    r.check_decode(1, heads_per_seq=[0, 5])


@pytest.mark.parametrize("d,dd,w,Hq,Hkv,lens", [
    (64, 16, 600, 8, 2, [30000, 1, 2, 0, 33, 700, 64, 100]),
    (128, 16, 100, 4, 2, [5, 9000, 0, 0, 1, 4000]),
    (64, 32, 48, 8, 2, [12000] + [3] * 20),
    (64, 16, 32, 4, 1, [7000, 10, 0, 2500]),
    (128, 32, 256, 8, 1, [1, 300, 6000]),
])
def test_mixed_lengths_equal_shares(d, dd, w, Hq, Hkv, lens):
    """The batch's cache bytes are dealt out in equal shares, one per
    workgroup: a long sequence beside tiny and empty ones is cut into many
    pieces (some boundaries fall inside a ring subtile), whose records the
    combine kernel merges; pairs a workgroup holds whole are finished there;
    empty sequences decode to NaN."""
    r = Ragged(WL.with_(d=d, dd=dd, w=w, Hq=Hq, Hkv=Hkv), lens, 64, steps=1)
    r.check_decode(0)
    r.append_step(0)
    r.check_decode(1)


def test_sequence_at_capacity_is_marked_overflowed():
    """A sequence whose blocks are all used stores nothing, is marked
    overflowed (lens = -1 - cap), stays so under a later append, and decodes
    to NaN; the other sequence appends and decodes as usual (oracle row)."""
    wl = WL.with_(w=16)
    r = Ragged(wl, [64, 10], 32, extra_blocks=0, steps=2)
    # sequence 0 holds exactly max_blocks * page_size tokens: fill it to capacity
    cap = r.pc.cap
    r.pc.lens[0] = cap
    before = raw(r.pc.k_pool).copy()
    k, v = r.step_tokens(0)
    dar.dar_cache_append_paged(r.pc, k, v, r.wdd, Hq=wl.Hq)
    torch.cuda.synchronize()
    assert r.pc.lens.cpu().tolist() == [-1 - cap, 11]
    assert r.pc.overflowed() == [0]
    # only sequence 1's page rows may have changed
    after = raw(r.pc.k_pool)
    changed = np.unique(np.nonzero((before != after).any(axis=(1, 2, 3)))[0])
    assert set(changed.tolist()) <= set(int(p) for p in r.bt[1] if p >= 0)
    k, v = r.step_tokens(1)
    dar.dar_cache_append_paged(r.pc, k, v, r.wdd, Hq=wl.Hq)
    torch.cuda.synchronize()
    assert r.pc.lens.cpu().tolist() == [-1 - cap, 12]
    assert np.array_equal(raw(r.pc.k_pool)[[p for p in r.bt[0] if p >= 0]],
                          before[[p for p in r.bt[0] if p >= 0]])
    g = np.random.Generator(np.random.PCG64(71))
    q = di.Tensor(g.standard_normal((2, wl.Hq, wl.d), dtype=np.float32), "bf16")
    o = to_host64(dar.dar_attn_decode_paged(r.pc, to_dev(q), r.wdd))
    assert np.isnan(o[0]).all()
    grp = wl.Hq // wl.Hkv
    for h in range(wl.Hq):
        gg = h // grp
        ref = oracle.rows(r.k[1].f64_slice(gg)[:12], r.v[1].f64_slice(gg)[:12], r.wd.f64[gg], None,
                          wl.w, [11], q.f64[1, h][None])
        assert np.abs(o[1, h] - ref[0]).max() <= tol("bf16")


@pytest.mark.parametrize("long_len", [100, 20000])
def test_empty_sequence_decodes_to_nan(long_len):
    """lens[b] = 0 (no query position): NaN rows for that sequence only, with
    one workgroup per (sequence, KV head) and with split records merged."""
    r = Ragged(WL, [long_len, 0, 37], 64, steps=1)
    g = np.random.Generator(np.random.PCG64(72))
    q = di.Tensor(g.standard_normal((3, WL.Hq, WL.d), dtype=np.float32), "bf16")
    o = to_host64(dar.dar_attn_decode_paged(r.pc, to_dev(q), r.wdd))
    assert np.isnan(o[1]).all()
    assert np.isfinite(o[0]).all() and np.isfinite(o[2]).all()


def test_full_size_ragged_decode1b():
    """decode1b shape (B32 Hq32 Hkv8 d64 d_down16 w512), lengths spread from
    1 to 32768 tokens, 256-token pages: sampled heads of every sequence."""
    wl = di.WORKLOADS["decode1b"]
    lens = [1, 2, 511, 512, 513] + [int(x) for x in np.linspace(1000, 32768, 27)]
    r = Ragged(wl, lens, 256, steps=1)
    r.check_decode(0, heads_per_seq=[0, 17, 31])
    r.append_step(0)
    r.check_decode(1, heads_per_seq=[4])


# ------------------------------------------------------------ rotary decode


def untied_wu(wl, seed=73):
    g = np.random.Generator(np.random.PCG64(seed))
    return di.Tensor(g.standard_normal((wl.Hkv, wl.dd, wl.d), dtype=np.float32) / np.sqrt(wl.dd),
                     "bf16")


@pytest.mark.parametrize("w,ps,r,untied", [(32, 64, 64, False), (0, 32, 16, True),
                                           (1, 256, 32, False), (600, 64, 16, False),
                                           (100, 32, 64, True)])
def test_rope_ragged_decode_and_append(w, ps, r, untied):
    """Ragged lengths (an empty sequence included): the rotary decode of
    every head of every sequence, appends in between."""
    wl = WL.with_(w=w)
    rg = Ragged(wl, [1, 37, 300, 0, 64, 511, 129], ps)
    rope = dar.Rope(r, 10000.0, n_pos=rg.pc.cap)
    wu = untied_wu(wl) if untied else None
    for t in range(2):
        rg.check_decode(t, rope=rope, wu=wu)
        rg.append_step(t)
    rg.check_decode(2, rope=rope, wu=wu)


@pytest.mark.parametrize("d,dd,G,r,untied", [(64, 32, 4, 32, False), (128, 16, 2, 16, True),
                                             (128, 32, 8, 64, False), (64, 16, 1, 64, True),
                                             (128, 32, 4, 32, True)])
def test_rope_other_shapes(d, dd, G, r, untied):
    wl = WL.with_(d=d, dd=dd, Hq=2 * G, Hkv=2, w=48)
    rg = Ragged(wl, [5, 200, 97, 0], 64)
    rope = dar.Rope(r, 500000.0, n_pos=rg.pc.cap + 7)
    wu = untied_wu(wl) if untied else None
    rg.check_decode(0, rope=rope, wu=wu)
    rg.append_step(0)
    rg.check_decode(1, rope=rope, wu=wu)


@pytest.mark.parametrize("d,dd,w,Hq,Hkv,lens,r", [
    (64, 16, 600, 8, 2, [30000, 1, 2, 0, 33, 700, 64, 100], 64),
    (128, 32, 256, 8, 1, [1, 300, 6000], 32),
    (64, 32, 48, 8, 2, [12000] + [3] * 20, 16),
])
def test_rope_mixed_lengths_split_pairs(d, dd, w, Hq, Hkv, lens, r):
    """A long sequence beside tiny and empty ones: its pairs are cut into
    many pieces whose records the combine merges (rotated distant keys in
    every piece at their own positions)."""
    rg = Ragged(WL.with_(d=d, dd=dd, w=w, Hq=Hq, Hkv=Hkv), lens, 64, steps=1)
    rope = dar.Rope(r, 10000.0 if d == 64 else 500000.0, n_pos=rg.pc.cap)
    rg.check_decode(0, rope=rope)
    rg.append_step(0)
    rg.check_decode(1, rope=rope)


def test_rope_zero_dim_equals_plain_paged_decode():
    """rotary_dim 0 rotates nothing: the output equals dar_attn_decode_paged's
    bit for bit."""
    rg = Ragged(WL.with_(w=64), [900, 1, 0, 333], 64, steps=1)
    g = np.random.Generator(np.random.PCG64(74))
    q = to_dev(di.Tensor(g.standard_normal((4, WL.Hq, WL.d), dtype=np.float32), "bf16"))
    a = dar.dar_attn_decode_paged(rg.pc, q, rg.wdd)
    b = dar.dar_attn_decode_paged_rope(rg.pc, q, rg.wdd, dar.Rope(0, 10000.0, n_pos=rg.pc.cap))
    torch.cuda.synchronize()
    assert np.array_equal(raw(a), raw(b))


def test_rope_overflowed_sequence_decodes_to_nan():
    """A sequence marked overflowed (lens = -1 - cap) decodes to NaN; the
    other one is served (oracle's rotary row)."""
    wl = WL.with_(w=16)
    rg = Ragged(wl, [64, 10], 32, extra_blocks=0, steps=1)
    cap = rg.pc.cap
    rg.pc.lens[0] = -1 - cap
    g = np.random.Generator(np.random.PCG64(75))
    q = di.Tensor(g.standard_normal((2, wl.Hq, wl.d), dtype=np.float32), "bf16")
    rope = dar.Rope(32, 10000.0, n_pos=cap)
    o = to_host64(dar.dar_attn_decode_paged_rope(rg.pc, to_dev(q), rg.wdd, rope))
    assert np.isnan(o[0]).all()
    grp = wl.Hq // wl.Hkv
    for h in range(wl.Hq):
        gg = h // grp
        ref = oracle.rows_rope(rg.k[1].f64_slice(gg)[:10], rg.v[1].f64_slice(gg)[:10], rg.wd.f64[gg],
                               None, wl.w, 32, 10000.0, 0, [9], q.f64[1, h][None])
        assert np.abs(o[1, h] - ref[0]).max() <= tol("bf16")


def test_rope_full_size_ragged_decode1b():
    """decode1b shape (B32 Hq32 Hkv8 d64 d_down16 w512) with rotary dimension
    64, lengths spread from 1 to 32768 tokens, 256-token pages: sampled heads
    of every sequence."""
    wl = di.WORKLOADS["decode1b"]
    lens = [1, 2, 511, 512, 513] + [int(x) for x in np.linspace(1000, 32768, 27)]
    rg = Ragged(wl, lens, 256, steps=1)
    rope = dar.Rope(64, 10000.0, n_pos=rg.pc.cap)
    rg.check_decode(0, heads_per_seq=[0, 17, 31], rope=rope)
    rg.append_step(0)
    rg.check_decode(1, heads_per_seq=[4], rope=rope)
