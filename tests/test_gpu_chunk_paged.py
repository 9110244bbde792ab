"""GPU chunked prefill over a paged split cache (dar_attn_prefill_chunk_paged
through the C ABI).

Sequences of different lengths share one batch; their latents live in pages
handed out through a shuffled block table. Each call gives sequence b its
own number of new tokens n_b (0 included) at its own position lens[b].
Checked against what the method fixes:
  * every written row of sequence b, and its log-sum-exp, equals the row at
    the same position of the oracle's prefill over that sequence alone
    (Eq. 3-4; tolerance 2e-2 for bf16 with fp32 accumulation), element by
    element; rows past n_b stay as they were (NaN), and the rows past n_b of
    q, k_new and v_new are NaN, so reading any of them would show;
  * afterwards every ring row and every latent page row of each sequence is
    byte-identical to a dense cache that dar_cache_append filled with the
    same tokens, and lens[b] has advanced by n_b;
  * a paged decode step after the chunks matches the oracle's row;
  * a sequence whose chunk does not fit is marked overflowed, gets NaN rows
    and keeps its cache, while the others are served.
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


class PagedChunks:
    """B sequences of `totals[b]` seeded N(0,1) tokens each (queries, keys,
    values), fed to a paged cache chunk by chunk; a shuffled block table
    covers each sequence's total (plus `extra_blocks` unmapped entries)."""

    def __init__(self, wl, totals, page_size, seed=900, untied=False, extra_blocks=1):
        self.wl, self.ps, self.B = wl, page_size, len(totals)
        self.totals = list(totals)
        g = np.random.Generator(np.random.PCG64(seed))
        self.wd = di.Tensor(g.standard_normal((wl.Hkv, wl.d, wl.dd), dtype=np.float32) /
                            np.sqrt(wl.d), "bf16")
        self.wu = (di.Tensor(g.standard_normal((wl.Hkv, wl.dd, wl.d), dtype=np.float32) /
                             np.sqrt(wl.dd), "bf16") if untied else None)
        self.q = [di.Tensor(g.standard_normal((wl.Hq, n, wl.d), dtype=np.float32), "bf16")
                  for n in totals]
        self.k = [di.Tensor(g.standard_normal((wl.Hkv, n, wl.d), dtype=np.float32), "bf16")
                  for n in totals]
        self.v = [di.Tensor(g.standard_normal((wl.Hkv, n, wl.d), dtype=np.float32), "bf16")
                  for n in totals]
        self.wdd, self.wud = to_dev(self.wd), to_dev(self.wu)
        self.qd = [to_dev(x) for x in self.q]
        self.kd = [to_dev(x) for x in self.k]
        self.vd = [to_dev(x) for x in self.v]
        nblk = [(n + page_size - 1) // page_size for n in totals]
        maxb = max(nblk) + extra_blocks
        n_pages = sum(nblk) + 3
        self.pc = dar.DarPagedCache(self.B, wl.Hkv, wl.d, wl.dd, wl.w, page_size, maxb, n_pages,
                                    torch.bfloat16)
        perm = g.permutation(n_pages)
        bt = np.full((self.B, maxb), -1, np.int32)
        nxt = 0
        for b, nb in enumerate(nblk):
            for blk in range(nb):
                bt[b, blk] = perm[nxt]
                nxt += 1
        self.bt = bt
        self.pc.block_table.copy_(torch.from_numpy(bt))
        self.lens = [0] * self.B
        self.ref = []
        for b in range(self.B):
            r, lse = oracle.prefill(self.q[b].f64[None], self.k[b].f64[None], self.v[b].f64[None],
                                    self.wd.f64, None if self.wu is None else self.wu.f64, wl.w,
                                    want_lse=True)
            self.ref.append((r[0], lse[0]))
        torch.cuda.synchronize()

    def chunk(self, nbs, n=None, pass_n_new=True):
        """One call: sequence b takes nbs[b] tokens (n the padded row count).
        Returns the max abs error over every written row."""
        wl = self.wl
        n = n or max(max(nbs), 1)
        nan = float("nan")
        q = torch.full((self.B, wl.Hq, n, wl.d), nan, dtype=torch.bfloat16, device="cuda")
        k = torch.full((self.B, wl.Hkv, n, wl.d), nan, dtype=torch.bfloat16, device="cuda")
        v = torch.full((self.B, wl.Hkv, n, wl.d), nan, dtype=torch.bfloat16, device="cuda")
        for b, nb in enumerate(nbs):
            L = self.lens[b]
            q[b, :, :nb] = self.qd[b][:, L:L + nb]
            k[b, :, :nb] = self.kd[b][:, L:L + nb]
            v[b, :, :nb] = self.vd[b][:, L:L + nb]
        o = torch.full((self.B, wl.Hq, n, wl.d), nan, dtype=torch.bfloat16, device="cuda")
        lse = torch.full((self.B, wl.Hq, n), nan, dtype=torch.float32, device="cuda")
        n_new = torch.tensor(nbs, dtype=torch.int32, device="cuda") if pass_n_new else None
        dar.dar_attn_prefill_chunk_paged(self.pc, q, k, v, self.wdd, w_up=self.wud, n_new=n_new,
                                         o=o, lse=lse)
        torch.cuda.synchronize()
        got = to_host64(o)
        gl = lse.double().cpu().numpy()
        worst = 0.0
        for b, nb in enumerate(nbs):
            L = self.lens[b]
            ref, ref_lse = self.ref[b]
            assert np.isnan(got[b, :, nb:]).all(), "rows past n_b were written (seq %d)" % b
            assert np.isnan(gl[b, :, nb:]).all()
            if nb == 0:
                continue
            assert np.isfinite(got[b, :, :nb]).all(), "seq %d: non-finite rows" % b
            err = np.abs(got[b, :, :nb] - ref[:, L:L + nb])
            assert err.max() <= tol("bf16"), "seq %d rows %d..%d: max abs err %.3g at %s" % (
                b, L, L + nb, err.max(), np.unravel_index(err.argmax(), err.shape))
            lerr = np.abs(gl[b, :, :nb] - ref_lse[:, L:L + nb]).max()
            assert lerr <= 2e-2, (b, lerr)
            worst = max(worst, float(err.max()))
            self.lens[b] = L + nb
        assert self.pc.lens.cpu().tolist() == self.lens
        return worst

    def check_cache(self):
        """Rings and latent pages against dense caches of the same tokens."""
        wl, ps = self.wl, self.ps
        for b, L in enumerate(self.lens):
            if L == 0:
                continue
            c = dar.DarCache(1, wl.Hkv, wl.d, wl.dd, wl.w, L, torch.bfloat16)
            dar.dar_cache_append(c, self.kd[b][None, :, :L].contiguous(),
                                 self.vd[b][None, :, :L].contiguous(), self.wdd, Hq=wl.Hq)
            torch.cuda.synchronize()
            if wl.w > 0:
                assert np.array_equal(raw(self.pc.k_win[b]), raw(c.k_win[0])), "ring keys of seq %d" % b
                assert np.array_equal(raw(self.pc.v_win[b]), raw(c.v_win[0])), "ring values of seq %d" % b
            for e0 in range(0, max(0, L - wl.w), ps):
                e1 = min(e0 + ps, L - wl.w)
                page = int(self.bt[b, e0 // ps])
                assert np.array_equal(raw(self.pc.k_pool[page, :, :e1 - e0]), raw(c.k_lat[0, :, e0:e1])), \
                    "latent keys of seq %d, positions %d..%d" % (b, e0, e1)
                assert np.array_equal(raw(self.pc.v_pool[page, :, :e1 - e0]), raw(c.v_lat[0, :, e0:e1])), \
                    "latent values of seq %d, positions %d..%d" % (b, e0, e1)

    def decode_step(self):
        """Append each sequence's next token and decode its next query."""
        wl = self.wl
        k = torch.stack([self.kd[b][:, self.lens[b]] for b in range(self.B)]).contiguous()
        v = torch.stack([self.vd[b][:, self.lens[b]] for b in range(self.B)]).contiguous()
        dar.dar_cache_append_paged(self.pc, k, v, self.wdd, Hq=wl.Hq)
        qd = torch.stack([self.qd[b][:, self.lens[b]] for b in range(self.B)]).contiguous()
        o = dar.dar_attn_decode_paged(self.pc, qd, self.wdd, w_up=self.wud)
        torch.cuda.synchronize()
        got = to_host64(o)
        for b in range(self.B):
            L = self.lens[b]
            err = np.abs(got[b] - self.ref[b][0][:, L]).max()
            assert err <= tol("bf16"), (b, err)
            self.lens[b] = L + 1


D64 = di.Workload("chunk_paged", 40, 4, 8, 2, 0, 64, 16, 32, "bf16")


@pytest.mark.parametrize("w", [0, 32, 100])
@pytest.mark.parametrize("ps", [32, 64])
def test_ragged_chunks(w, ps):
    """Three calls with a different token count per sequence (0 and 1
    included), from an empty cache; then the caches and a decode step."""
    plan = [[70, 1, 0, 200], [33, 64, 5, 0], [1, 130, 64, 41]]
    totals = [sum(c[b] for c in plan) + 1 for b in range(4)]
    pc = PagedChunks(D64.with_(w=w), totals, ps, untied=(w == 32))
    for nbs in plan:
        pc.chunk(nbs)
    pc.check_cache()
    pc.decode_step()


@pytest.mark.parametrize("d,dd,w,ps", [(64, 32, 48, 32), (128, 16, 64, 64), (128, 32, 200, 128),
                                       (128, 32, 0, 32)])
def test_other_shapes(d, dd, w, ps):
    wl = di.Workload("chunk_paged_%d_%d" % (d, dd), 41, 3, 8, 4, 0, d, dd, w, "bf16")
    plan = [[150, 40, 97], [64, 129, 3], [31, 0, 200]]
    totals = [sum(c[b] for c in plan) + 1 for b in range(3)]
    pc = PagedChunks(wl, totals, ps, untied=(dd == 32))
    for nbs in plan:
        pc.chunk(nbs)
    pc.check_cache()
    pc.decode_step()


def test_uniform_chunks_without_n_new():
    """n_new omitted: every sequence takes n tokens; sequences that start at
    different lengths (a ragged prefix first)."""
    plan = [[300, 17, 129], [64, 64, 64], [64, 64, 64]]
    totals = [sum(c[b] for c in plan) + 1 for b in range(3)]
    pc = PagedChunks(D64.with_(w=64, B=3), totals, 32)
    pc.chunk(plan[0])
    pc.chunk(plan[1], pass_n_new=False)
    pc.chunk(plan[2], pass_n_new=False)
    pc.check_cache()
    pc.decode_step()


def test_overflow_marks_sequence():
    """Sequence 1's chunk does not fit its block table (capacity 224 tokens):
    its rows are NaN, lens becomes -1 - len, its cache is unchanged; the
    other sequences are served."""
    wl = D64.with_(w=32, B=3)
    pc = PagedChunks(wl, [200, 200, 200], 32, extra_blocks=0)
    pc.chunk([60, 60, 60])
    cap = pc.pc.cap
    ring_before = raw(pc.pc.k_win[1]).copy()
    pool_before = raw(pc.pc.k_pool).copy()
    nan = float("nan")
    n = cap
    q = torch.full((3, wl.Hq, n, wl.d), nan, dtype=torch.bfloat16, device="cuda")
    k = torch.full((3, wl.Hkv, n, wl.d), nan, dtype=torch.bfloat16, device="cuda")
    v = torch.full((3, wl.Hkv, n, wl.d), nan, dtype=torch.bfloat16, device="cuda")
    nbs = [10, cap - 60 + 1, 0]
    for b in (0, 1):
        q[b, :, :nbs[b]] = pc.qd[b][:, 60:60 + nbs[b]] if b == 0 else 0.5
        k[b, :, :nbs[b]] = pc.kd[b][:, 60:60 + nbs[b]] if b == 0 else 0.5
        v[b, :, :nbs[b]] = pc.vd[b][:, 60:60 + nbs[b]] if b == 0 else 0.5
    o = torch.full_like(q, nan)
    dar.dar_attn_prefill_chunk_paged(pc.pc, q, k, v, pc.wdd, n_new=torch.tensor(nbs, dtype=torch.int32,
                                                                                  device="cuda"), o=o)
    torch.cuda.synchronize()
    assert pc.pc.lens.cpu().tolist() == [70, -1 - 60, 60]
    got = to_host64(o)
    assert np.isnan(got[1]).all()
    assert np.abs(got[0, :, :10] - pc.ref[0][0][:, 60:70]).max() <= tol("bf16")
    assert np.isnan(got[2]).all()
    assert np.array_equal(raw(pc.pc.k_win[1]), ring_before), "overflowed sequence's ring changed"
    pool_after = raw(pc.pc.k_pool)
    for blk in range(pc.bt.shape[1]):
        page = pc.bt[1, blk]
        if page >= 0:
            assert np.array_equal(pool_after[page], pool_before[page]), "overflowed sequence's pages changed"


def test_full_size_decode1b_heads():
    """The 1B-decode head layout (Hq 32, Hkv 8, d 64, d_down 16, w 512) with
    histories of 2-6K tokens and a 256-token chunk per sequence: every row of
    two KV heads' query groups per sequence against the oracle's rows over the
    sequence's whole history (output NaN-filled first)."""
    wl = di.Workload("chunk_paged_1b", 42, 4, 32, 8, 0, 64, 16, 512, "bf16")
    hist = [2048, 6000, 3333, 4100]
    n = 256
    g = np.random.Generator(np.random.PCG64(43))
    ps = 64
    tot = [L + n for L in hist]
    k = [di.Tensor(g.standard_normal((wl.Hkv, t, wl.d), dtype=np.float32), "bf16") for t in tot]
    v = [di.Tensor(g.standard_normal((wl.Hkv, t, wl.d), dtype=np.float32), "bf16") for t in tot]
    q = di.Tensor(g.standard_normal((4, wl.Hq, n, wl.d), dtype=np.float32), "bf16")
    wd = di.Tensor(g.standard_normal((wl.Hkv, wl.d, wl.dd), dtype=np.float32) / 8.0, "bf16")
    wdd = to_dev(wd)
    maxb = max((t + ps - 1) // ps for t in tot)
    n_pages = 4 * maxb + 1
    pc = dar.DarPagedCache(4, wl.Hkv, wl.d, wl.dd, wl.w, ps, maxb, n_pages, torch.bfloat16)
    perm = g.permutation(n_pages)
    bt = perm[:4 * maxb].reshape(4, maxb).astype(np.int32)
    pc.block_table.copy_(torch.from_numpy(bt))
    kd = [to_dev(x) for x in k]
    vd = [to_dev(x) for x in v]
    # histories through the chunk path itself (n_new = each history length)
    Lmax = max(hist)
    kh = torch.zeros(4, wl.Hkv, Lmax, wl.d, dtype=torch.bfloat16, device="cuda")
    vh = torch.zeros_like(kh)
    for b, L in enumerate(hist):
        kh[b, :, :L] = kd[b][:, :L]
        vh[b, :, :L] = vd[b][:, :L]
    qh = torch.zeros(4, wl.Hq, Lmax, wl.d, dtype=torch.bfloat16, device="cuda")
    dar.dar_attn_prefill_chunk_paged(pc, qh, kh, vh, wdd,
                                     n_new=torch.tensor(hist, dtype=torch.int32, device="cuda"))
    kn = torch.stack([kd[b][:, hist[b]:] for b in range(4)]).contiguous()
    vn = torch.stack([vd[b][:, hist[b]:] for b in range(4)]).contiguous()
    o = torch.full((4, wl.Hq, n, wl.d), float("nan"), dtype=torch.bfloat16, device="cuda")
    dar.dar_attn_prefill_chunk_paged(pc, to_dev(q), kn, vn, wdd, o=o)
    torch.cuda.synchronize()
    assert pc.lens.cpu().tolist() == tot
    got = to_host64(o)
    assert np.isfinite(got).all()
    grp = wl.Hq // wl.Hkv
    worst = 0.0
    for b, L in enumerate(hist):
        rows = np.arange(L, L + n)
        for gg in (b % wl.Hkv, (b + 5) % wl.Hkv):
            hs = list(range(gg * grp, (gg + 1) * grp))
            qr = q.f64[b, hs].reshape(-1, wl.d)
            ref = oracle.rows(k[b].f64[gg], v[b].f64[gg], wd.f64[gg], None, wl.w, np.tile(rows, grp), qr)
            worst = max(worst, float(np.abs(got[b, hs].reshape(-1, wl.d) - ref).max()))
    print("[chunk paged] max abs err %.4g" % worst, flush=True)
    assert worst <= tol("bf16"), worst
