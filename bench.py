"""DAR attention benchmark on one MI355X.

One step = the whole hot path once:
  * causal prefill of the Pythia-70M-shaped batch (B8 H8 T2048 d64 d_down16
    w256, bf16): window-exit latent pre-pass + two-region attention kernel;
  * one decode step of the 1B-scale batch over its split cache (B32 Hq32
    Hkv8 d64 d_down16 w512, 32768 cached tokens): cache append of the new
    token (window exit projected to its latent) + split-KV decode.
Inputs are seeded synthetic N(0,1) tensors of those shapes, resident in HBM
before timing starts. `ms_per_step` times whole steps back to back; then each
operation is timed on its own over the same number of back-to-back calls (the
decode at the final cache length, which it does not change), with one event
pair around each run. `value` is the prefill's algorithmic TFLOP/s; the decode
KV GB/s is reported beside it. The backward of the same prefill (the training
step's attention part, given the forward's output and log-sum-exp) is timed
the same way and reported under "backward".

Also reported, each timed the same way: the prefill and the decode with a
cold cache hierarchy (a 1 GiB buffer written between calls evicts L2 and
the Infinity Cache; the time of the writes alone is subtracted), the prefill
and the decode with the rotary embedding inside Eq. 3 (prefill: rotary
dimension 16 of 64, base 10000, as in the Pythia models; decode: full
rotation), the prefill and the decode with a single shared latent per token
(the same batches, with seeded N(0,1) latents and N(0, 1/d_down) U_K, U_V:
the decode streams one latent array instead of two), the decode over a
paged cache (256-token pages in shuffled order; every sequence at the decode
length, then lengths spread from 1K to 32K tokens: a ragged batch), the
chunked prefill and the other prefill workloads.

Prints ONE JSON line (rank 0). Only one GPU is used: --gpus above 1 exits.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E
# The exponential ceiling (v_exp_f32 results per second for the whole device,
# at the clock the device holds under that load) is measured at the start of
# every run by the machine microbenchmarks (paper_2606_18587_amd/k0.py,
# include/dar_k0.h) and reported under "k0".
ROPE_PREFILL_DIM = 16       # rotary dimension of the prefill line (Pythia: 25% of 64)
ROPE_DECODE_DIM = 64        # full rotation on the decode line
ROPE_BASE = 10000.0

# HBM bytes per entry-point launch from two rocprofv3 counter runs (FETCH_SIZE,
# then WRITE_SIZE), each scaled by what the counter reads for a plain 256 MiB
# device copy (profiles/hbm_traffic_prefill_pythia70m_decode1b.md). A record
# holds only while the kernel sources it was taken on are unchanged: their
# hash is checked at run time and the traffic is reported as null otherwise.
CSRC = os.path.join(ROOT, "paper_2606_18587_amd", "csrc")
MEASURED_TRAFFIC = {
    "prefill": {"files": ["dar_api.hip", "dar_common.hpp", "dar_kernels.hpp", "latent.hip",
                          "prefill_mfma.hip"],
                "sha256_16": "78f2401ce7252071", "bytes": 126117468},
    "decode": {"files": ["dar_api.hip", "dar_common.hpp", "dar_kernels.hpp", "decode.hip",
                         "decode_mfma.hip"],
               "sha256_16": "6556aad07ed64880", "bytes": 563628767},
    "backward": {"files": ["dar_api.hip", "dar_common.hpp", "dar_kernels.hpp", "mfma_common.hpp",
                           "backward.hip", "backward_mfma.hip"],
                 "sha256_16": "a2ed4e6dfcfdec0a", "bytes": 502792476},
}


def measured_traffic(which):
    """Counter-derived HBM bytes per launch, or None if the sources changed."""
    import hashlib

    rec = MEASURED_TRAFFIC[which]
    m = hashlib.sha256()
    for f in rec["files"]:
        with open(os.path.join(CSRC, f), "rb") as fh:
            m.update(fh.read())
    return rec["bytes"] if m.hexdigest()[:16] == rec["sha256_16"] else None


def head_start(torch, steps):
    """Keep the GPU busy (a spin kernel on the current stream, ahead of the
    first timed event) while the host enqueues every timed step, so that the
    per-call events measure GPU execution and not the Python launch path
    (about 50 us per step of ctypes marshalling, more than a prefill lasts).
    The spin is outside the timed region; 1 ms of head start per step."""
    torch.cuda._sleep(int(2.4e9 * 1e-3 * steps))


CHUNK_N = 256       # new tokens per chunked-prefill call
CHUNK_CALLS = 5     # timed chunked-prefill calls


def chunk_flops(B, Hq, L, n, d, dd, w):
    """Rows L..L+n-1 of a causal prefill: 4 d flop per window pair, 4 d_down
    per distant pair."""
    i = np.arange(L, L + n, dtype=np.int64)
    nl = np.minimum(i + 1, w).sum()
    nd = (i + 1).sum() - nl
    return float(B * Hq * (4 * d * nl + 4 * dd * nd))


def prefill_flops(B, Hq, T, d, dd, w):
    """Algorithmic flops: QK^T and PV at 2 flop/MAC, d wide inside the window,
    d_down wide beyond it; masked and skipped work is not counted."""
    i = np.arange(T, dtype=np.int64)
    n_loc = np.minimum(i + 1, w).sum()
    n_dist = (i + 1).sum() - n_loc
    return float(B * Hq * (4 * d * n_loc + 4 * dd * n_dist))


def backward_flops(B, Hq, T, d, dd, w):
    """Algorithmic flops of the prefill backward at 2 flop/MAC: per window pair
    the five d-wide products (S, dP recomputed; dV, dK, dQ), per distant pair
    the six d_down-wide ones (S, dP; gK, gV to the keys; h and the latent
    output to the queries). The O(T d d_down) projections and lifts are not
    counted."""
    i = np.arange(T, dtype=np.int64)
    n_loc = np.minimum(i + 1, w).sum()
    n_dist = (i + 1).sum() - n_loc
    return float(B * Hq * (10 * d * n_loc + 12 * dd * n_dist))


def full_backward_flops(B, Hq, T, d):
    """Algorithmic flops of the backward with the rotary embedding: every
    causal pair at full d (the distant keys are lifted and rotated), five
    d-wide products per pair (S, dP recomputed; dV, dK, dQ) at 2 flop/MAC."""
    return float(B * Hq * (T * (T + 1) // 2) * 10 * d)


def decode_bytes_shared(B, Hq, Hkv, d, dd, w, L, esize=2):
    """As decode_bytes with one shared latent per token (one latent stream
    for keys and values), plus the two U matrices."""
    n_win = min(L, w)
    n_lat = L - n_win
    kv = B * Hkv * (2 * n_win * d + n_lat * dd) * esize
    return float(kv + 2 * B * Hq * d * esize + 2 * Hkv * d * dd * esize)


def full_flops(B, Hq, T, d):
    """Causal attention at d for every pair (the rotary path: distant keys are
    lifted to full d, Eq. 3): 4 d flop per pair."""
    return float(B * Hq * 4 * d * (T * (T + 1) // 2))


def decode_bytes(B, Hq, Hkv, d, dd, w, L, esize=2):
    """Algorithmic HBM bytes of one decode step at cache length L: ring and
    latents (keys and values) once, plus query, output and W_down."""
    n_win = min(L, w)
    n_lat = L - n_win
    kv = B * Hkv * 2 * (n_win * d + n_lat * dd) * esize
    return float(kv + 2 * B * Hq * d * esize + Hkv * d * dd * esize)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-backward", action="store_true",
                    help="skip the separately timed prefill backward")
    ap.add_argument("--no-chunk", action="store_true",
                    help="skip the chunked prefill into the decode cache")
    ap.add_argument("--no-other-prefill", action="store_true",
                    help="skip the prefill workloads reported beside the main one")
    ap.add_argument("--no-rope", action="store_true",
                    help="skip the prefill and decode with the rotary embedding")
    ap.add_argument("--no-ragged", action="store_true",
                    help="skip the ragged-batch prefill line")
    ap.add_argument("--no-paged", action="store_true",
                    help="skip the decode over a paged cache")
    ap.add_argument("--no-shared", action="store_true",
                    help="skip the prefill and decode with a single shared latent")
    ap.add_argument("--no-cold", action="store_true",
                    help="skip the cold-cache timings")
    ap.add_argument("--no-launch", action="store_true",
                    help="skip the host launch-cost and graph-replay measurement")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain device copy of known size (HBM counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU only; the library has no multi-GPU path "
              "(run with --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import torch

    import dar_inputs as di
    import paper_2606_18587_amd as dar

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.copy_calibration:
        copy_calibration(torch, dev)
        return
    from paper_2606_18587_amd import k0 as k0_bench

    k0 = k0_bench.measure(dev)

    def up(t):
        if t is None:
            return None
        if t.dtype == "bf16":
            return torch.from_numpy(t.store.view(np.int16)).view(torch.bfloat16).to(dev)
        return torch.from_numpy(t.store).to(dev)

    # ---------------- prefill workload
    pw = di.WORKLOADS["pythia70m"]
    pin = di.make_prefill_inputs(pw)
    q, k, v, wd = (up(pin[x]) for x in ("q", "k", "v", "wd"))
    o = torch.empty_like(q)
    shape = dar.make_shape(pw.B, pw.Hq, pw.Hkv, pw.d, pw.dd, pw.w, torch.bfloat16)
    ws = torch.empty(max(1, dar.dar_prefill_workspace_bytes(shape, pw.T)), dtype=torch.uint8,
                     device=dev)
    flops = prefill_flops(pw.B, pw.Hq, pw.T, pw.d, pw.dd, pw.w)

    # ---------------- decode workload
    dw = di.WORKLOADS["decode1b"]
    t0 = time.time()
    pre = di.make_decode_prefix(dw, dw.T)
    cap = dw.T + args.warmup + 2 * args.steps + 1 + (CHUNK_CALLS + 1) * CHUNK_N
    cache = dar.DarCache(dw.B, dw.Hkv, dw.d, dw.dd, dw.w, cap, torch.bfloat16, device=dev)
    dwd = up(pre["wd"])
    kpre, vpre = up(pre["k"]), up(pre["v"])
    del pre
    dar.dar_cache_append(cache, kpre, vpre, dwd, Hq=dw.Hq)
    # the same tokens in a single-shared-latent cache, with seeded latents
    scache = None
    if not args.no_shared:
        gs = torch.Generator(device=dev).manual_seed(260618588)
        scache = dar.DarCache(dw.B, dw.Hkv, dw.d, dw.dd, dw.w, dw.T, torch.bfloat16, device=dev,
                              shared=True)
        clat = torch.randn(dw.B, dw.Hkv, dw.T, dw.dd, device=dev, generator=gs).bfloat16()
        dar.dar_cache_append_shared(scache, kpre, vpre, clat, Hq=dw.Hq)
        s_uk = (torch.randn(dw.Hkv, dw.dd, dw.d, device=dev, generator=gs) / dw.dd ** 0.5).bfloat16()
        s_uv = (torch.randn(dw.Hkv, dw.dd, dw.d, device=dev, generator=gs) / dw.dd ** 0.5).bfloat16()
        del clat
    del kpre, vpre
    dshape = dar.make_shape(dw.B, dw.Hq, dw.Hkv, dw.d, dw.dd, dw.w, torch.bfloat16)
    dws = torch.empty(dar.dar_decode_workspace_bytes(dshape, cap), dtype=torch.uint8, device=dev)
    n_step_inputs = args.warmup + args.steps
    step_in = []
    for t in range(n_step_inputs):
        st = di.make_decode_step(dw, t)
        step_in.append((up(st["q"]), up(st["k"]), up(st["v"])))
    dout = torch.empty(dw.B, dw.Hq, dw.d, dtype=torch.bfloat16, device=dev)
    torch.cuda.synchronize()
    setup_s = time.time() - t0

    def one_step(idx):
        qd, kd, vd = step_in[idx]
        dar.dar_attn_prefill(q, k, v, wd, None, pw.w, o=o, ws=ws, check=False)
        dar.dar_cache_append(cache, kd, vd, dwd, Hq=dw.Hq)
        dar.dar_attn_decode(cache, qd, dwd, None, o=dout, ws=dws)

    def timed(fn, n):
        """Mean GPU time (ms) of n back-to-back calls of fn(i): one event pair
        around the whole run (an event marker between two kernels costs the
        stream several microseconds of idle time, more than a cache append)."""
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        head_start(torch, n)
        e0.record()
        for i in range(n):
            fn(i)
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / n

    for i in range(args.warmup):
        one_step(i)
    torch.cuda.synchronize()

    # whole steps (prefill + append + decode), then each operation on its own
    L_first = cache.len + 1
    step_ms = timed(lambda i: one_step(args.warmup + i), args.steps)
    L_last = cache.len
    total_ms = step_ms * args.steps
    pre_ms = timed(lambda i: dar.dar_attn_prefill(q, k, v, wd, None, pw.w, o=o, ws=ws, check=False),
                   args.steps)
    qd_last = step_in[-1][0]
    dec_ms = timed(lambda i: dar.dar_attn_decode(cache, qd_last, dwd, None, o=dout, ws=dws),
                   args.steps)
    app_ms = timed(lambda i: dar.dar_cache_append(cache, step_in[i][1], step_in[i][2], dwd,
                                                  Hq=dw.Hq), args.steps)

    # cold cache hierarchy: a 1 GiB write between calls; the writes alone are
    # timed the same way and subtracted
    cold = {}
    if not args.no_cold:
        flushbuf = torch.empty(1 << 30, dtype=torch.uint8, device=dev)

        def timed_cold(fn, n):
            both = timed(lambda i: (flushbuf.fill_(i & 0xff), fn(i)), n)
            alone = timed(lambda i: flushbuf.fill_(i & 0xff), n)
            return both - alone

        cold["prefill_ms"] = timed_cold(
            lambda i: dar.dar_attn_prefill(q, k, v, wd, None, pw.w, o=o, ws=ws, check=False),
            args.steps)
        cold["decode_ms"] = timed_cold(
            lambda i: dar.dar_attn_decode(cache, qd_last, dwd, None, o=dout, ws=dws), args.steps)
        del flushbuf

    # single shared latent: the prefill batch with seeded latents, and the
    # decode over the shared cache (query at its last position)
    shared = {}
    if scache is not None:
        gp = torch.Generator(device=dev).manual_seed(260618589)
        pc = torch.randn(pw.B, pw.Hkv, pw.T, pw.dd, device=dev, generator=gp).bfloat16()
        p_uk = (torch.randn(pw.Hkv, pw.dd, pw.d, device=dev, generator=gp) / pw.dd ** 0.5).bfloat16()
        p_uv = (torch.randn(pw.Hkv, pw.dd, pw.d, device=dev, generator=gp) / pw.dd ** 0.5).bfloat16()
        run_sp = lambda i: dar.dar_attn_prefill_shared(q, k, v, pc, p_uk, p_uv, pw.w, o=o, ws=ws)
        for i in range(args.warmup):
            run_sp(i)
        shared["prefill_ms"] = timed(run_sp, args.steps)
        del pc
        run_sd = lambda i: dar.dar_attn_decode_shared(scache, qd_last, s_uk, s_uv, o=dout, ws=dws)
        for i in range(args.warmup):
            run_sd(i)
        shared["decode_ms"] = timed(run_sd, args.steps)
        shared["decode_len"] = scache.len
        del scache

    # ragged prefill: the same padded batch, sequence lengths spread evenly
    # over 256..T in a seeded order
    ragged = {}
    if not args.no_ragged:
        lens_p = torch.linspace(256, pw.T, pw.B).round().to(torch.int32)
        lens_p = lens_p[torch.randperm(pw.B, generator=torch.Generator().manual_seed(260618592))]
        sl_dev = lens_p.to(dev)
        run_rg = lambda i: dar.dar_attn_prefill_ragged(q, k, v, wd, None, pw.w, sl_dev, o=o, ws=ws)
        for i in range(args.warmup):
            run_rg(i)
        ragged["ms"] = timed(run_rg, args.steps)
        ragged["lens"] = [int(x) for x in lens_p.tolist()]

    # paged cache: the decode cache's contents copied into 256-token pages
    # handed out in a seeded random order; then the same pages with ragged
    # lengths (the sequences' first tokens only)
    paged = {}
    if not args.no_paged:
        PS = 256
        L = cache.len
        nblk = (L + 1 + PS - 1) // PS
        n_pages = dw.B * nblk
        pcache = dar.DarPagedCache(dw.B, dw.Hkv, dw.d, dw.dd, dw.w, PS, nblk, n_pages,
                                   torch.bfloat16, device=dev)
        perm = torch.randperm(n_pages, generator=torch.Generator().manual_seed(260618590))
        bt = perm.view(dw.B, nblk).to(torch.int32)
        pcache.block_table.copy_(bt)
        pcache.k_win.copy_(cache.k_win)
        pcache.v_win.copy_(cache.v_win)
        n_lat = L - dw.w
        for blk in range(nblk):
            e0, e1 = blk * PS, min((blk + 1) * PS, n_lat)
            if e1 <= e0:
                break
            pages = bt[:, blk].long().to(dev)
            pcache.k_pool[pages, :, : e1 - e0] = cache.k_lat[:, :, e0:e1]
            pcache.v_pool[pages, :, : e1 - e0] = cache.v_lat[:, :, e0:e1]
        pcache.lens.fill_(L)
        run_pd = lambda i: dar.dar_attn_decode_paged(pcache, qd_last, dwd, o=dout, ws=dws)
        for i in range(args.warmup):
            run_pd(i)
        paged["uniform_ms"] = timed(run_pd, args.steps)
        paged["uniform_len"] = L
        lens_r = torch.linspace(1024, L, dw.B).round().to(torch.int32)
        lens_r = lens_r[torch.randperm(dw.B, generator=torch.Generator().manual_seed(260618591))]
        pcache.lens.copy_(lens_r)
        for i in range(args.warmup):
            run_pd(i)
        paged["ragged_ms"] = timed(run_pd, args.steps)
        paged["ragged_lens"] = [int(x) for x in lens_r.tolist()]
        if not args.no_rope:
            # the same ragged batch with the rotary embedding of Eq. 3
            rpg = dar.Rope(ROPE_DECODE_DIM, ROPE_BASE, n_pos=pcache.cap, device=dev)
            run_pr = lambda i: dar.dar_attn_decode_paged_rope(pcache, qd_last, dwd, rpg, o=dout,
                                                              ws=dws)
            for i in range(args.warmup):
                run_pr(i)
            paged["ragged_rope_ms"] = timed(run_pr, args.steps)
        # skewed: one sequence at full length, the others at 600 tokens
        lens_s = [L] + [600] * (dw.B - 1)
        pcache.lens.copy_(torch.tensor(lens_s, dtype=torch.int32))
        for i in range(args.warmup):
            run_pd(i)
        paged["skewed_ms"] = timed(run_pd, args.steps)
        paged["skewed_lens"] = lens_s
        del pcache

    # the rotary embedding inside Eq. 3: the same prefill batch (un-rotated
    # queries and keys) and the same decode cache
    rope = {}
    if not args.no_rope:
        rp = dar.Rope(ROPE_PREFILL_DIM, ROPE_BASE, n_pos=pw.T, device=dev)
        rws = torch.empty(dar.dar_prefill_rope_workspace_bytes(shape, pw.T), dtype=torch.uint8,
                          device=dev)
        run_rp = lambda i: dar.dar_attn_prefill_rope(q, k, v, wd, None, pw.w, rp, o=o, ws=rws,
                                                     check=False)
        for i in range(args.warmup):
            run_rp(i)
        rope["prefill_ms"] = timed(run_rp, args.steps)
        del rws
        rd = dar.Rope(ROPE_DECODE_DIM, ROPE_BASE, n_pos=cap, device=dev)
        run_rd = lambda i: dar.dar_attn_decode_rope(cache, qd_last, dwd, rd, o=dout, ws=dws)
        for i in range(args.warmup):
            run_rd(i)
        rope["decode_ms"] = timed(run_rd, args.steps)
        # d = 128 heads: a cache of the long16k shape (batch 8) filled with
        # seeded N(0,1) ring entries and latents, the plain decode beside it
        B8, H8, K8, D8, DD8, W8, L8 = 8, 32, 8, 128, 32, 1024, 16384
        g8 = torch.Generator(device=dev).manual_seed(260618593)
        c8 = dar.DarCache(B8, K8, D8, DD8, W8, L8, torch.bfloat16, device=dev)
        for t in (c8.k_win, c8.v_win, c8.k_lat, c8.v_lat):
            t.copy_(torch.randn(t.shape, device=dev, generator=g8))
        c8.struct.len = L8
        q8 = torch.randn(B8, H8, D8, device=dev, generator=g8).bfloat16()
        wd8 = (torch.randn(K8, D8, DD8, device=dev, generator=g8) / D8 ** 0.5).bfloat16()
        o8 = torch.empty_like(q8)
        sh8 = dar.make_shape(B8, H8, K8, D8, DD8, W8, torch.bfloat16)
        ws8 = torch.empty(dar.dar_decode_workspace_bytes(sh8, L8), dtype=torch.uint8, device=dev)
        rd8 = dar.Rope(ROPE_DECODE_DIM, ROPE_BASE, n_pos=L8, device=dev)
        run_r8 = lambda i: dar.dar_attn_decode_rope(c8, q8, wd8, rd8, o=o8, ws=ws8)
        run_p8 = lambda i: dar.dar_attn_decode(c8, q8, wd8, None, o=o8, ws=ws8)
        for i in range(args.warmup):
            run_r8(i)
            run_p8(i)
        rope["d128_decode_ms"] = timed(run_r8, args.steps)
        rope["d128_plain_ms"] = timed(run_p8, args.steps)
        rope["d128_bytes"] = decode_bytes(B8, H8, K8, D8, DD8, W8, L8)
        del c8, ws8

    # chunked prefill into the same decode cache: chunks of CHUNK_N new tokens
    # (seeded N(0,1) queries, keys and values; the same tensors each call, at
    # advancing positions) attend to the ring, the latents and each other
    chunk = None
    if not args.no_chunk:
        gc = torch.Generator(device=dev).manual_seed(260618587)
        cq = torch.randn(dw.B, dw.Hq, CHUNK_N, dw.d, device=dev, generator=gc).bfloat16()
        ck = torch.randn(dw.B, dw.Hkv, CHUNK_N, dw.d, device=dev, generator=gc).bfloat16()
        cv = torch.randn(dw.B, dw.Hkv, CHUNK_N, dw.d, device=dev, generator=gc).bfloat16()
        co = torch.empty_like(cq)
        n_chunk = CHUNK_CALLS
        cws = torch.empty(dar.dar_prefill_chunk_workspace_bytes(
            dshape, cache.len + (n_chunk + 1) * CHUNK_N, CHUNK_N), dtype=torch.uint8, device=dev)
        run_chunk = lambda i: dar.dar_attn_prefill_chunk(cache, cq, ck, cv, dwd, None, o=co, ws=cws,
                                                         check=False)
        run_chunk(0)  # warm-up
        L0 = cache.len
        ch_ms = timed(run_chunk, n_chunk)
        cfl = np.mean([chunk_flops(dw.B, dw.Hq, L0 + c * CHUNK_N, CHUNK_N, dw.d, dw.dd, dw.w)
                       for c in range(n_chunk)])
        ctf = cfl / (ch_ms * 1e-3) / 1e12
        chunk = {"shape": "B%d Hq%d Hkv%d d%d d_down%d w%d, %d new tokens per call" % (
                     dw.B, dw.Hq, dw.Hkv, dw.d, dw.dd, dw.w, CHUNK_N),
                 "cache_len": [L0, cache.len], "us": round(ch_ms * 1e3, 1),
                 "tflops": round(ctf, 2), "frac_bf16_peak": round(ctf / PEAK_BF16_TFLOPS, 4),
                 "alg_flop": cfl}
        # the same chunks through the paged cache: a paged copy of the cache as
        # the dense calls left it (64-token pages, identity block table), each
        # sequence taking CHUNK_N tokens per call
        ps = 64
        maxb = (cache.cap + ps - 1) // ps
        pcache = dar.DarPagedCache(dw.B, dw.Hkv, dw.d, dw.dd, dw.w, ps, maxb, dw.B * maxb,
                                   torch.bfloat16)
        for src, dst in ((cache.k_lat, pcache.k_pool), (cache.v_lat, pcache.v_pool)):
            full = torch.zeros(dw.B, dw.Hkv, maxb * ps, dw.dd, dtype=torch.bfloat16, device=dev)
            full[:, :, :cache.cap] = src
            dst.copy_(full.view(dw.B, dw.Hkv, maxb, ps, dw.dd).permute(0, 2, 1, 3, 4)
                      .reshape(dw.B * maxb, dw.Hkv, ps, dw.dd))
            del full
        pcache.k_win.copy_(cache.k_win)
        pcache.v_win.copy_(cache.v_win)
        pcache.block_table.copy_(torch.arange(dw.B * maxb, dtype=torch.int32, device=dev)
                                 .view(dw.B, maxb))
        Lp = max(0, cache.cap - (n_chunk + 1) * CHUNK_N)
        Lp = min(Lp, cache.len)
        pcache.lens.fill_(Lp)
        pws = torch.empty(dar.dar_prefill_chunk_paged_workspace_bytes(dshape, pcache.cap, CHUNK_N),
                          dtype=torch.uint8, device=dev)
        run_pchunk = lambda i: dar.dar_attn_prefill_chunk_paged(pcache, cq, ck, cv, dwd, o=co, ws=pws)
        run_pchunk(0)  # warm-up
        pch_ms = timed(run_pchunk, n_chunk)
        pfl = np.mean([chunk_flops(dw.B, dw.Hq, Lp + (c + 1) * CHUNK_N, CHUNK_N, dw.d, dw.dd, dw.w)
                       for c in range(n_chunk)])
        chunk["paged"] = {"page_size": ps, "cache_len": [Lp + CHUNK_N, Lp + (n_chunk + 1) * CHUNK_N],
                          "us": round(pch_ms * 1e3, 1),
                          "tflops": round(pfl / (pch_ms * 1e-3) / 1e12, 2)}
        del pcache, pws, cws, cq, ck, cv, co

    pre_us = float(pre_ms * 1e3)
    dec_us = float(dec_ms * 1e3)
    tflops = flops / (pre_us * 1e-6) / 1e12
    dbytes = decode_bytes(dw.B, dw.Hq, dw.Hkv, dw.d, dw.dd, dw.w, L_last)
    gbs = dbytes / (dec_us * 1e-6) / 1e9

    # ---------------- the other prefill workloads (the parity-test shapes of
    # the other prefill configurations), each timed the same way; not part of `value`
    other = {}
    if not args.no_other_prefill:
        # pythia70m_dd32: the same batch with d_down 32, the distant width of the
        # decoupled-rotary cache the paper's Limitations section names (latent
        # 16 + an uncompressed rotary key part of 16, the Pythia rotary width):
        # the cost of absorbing W_up with a rotary model, against the rotary
        # line below that lifts the distant keys to full d
        for name in ("pythia410m_w128", "pythia410m_w512", "long16k", "pythia70m_dd32"):
            ow_ = (di.WORKLOADS["pythia70m"].with_(name=name, dd=32) if name == "pythia70m_dd32"
                   else di.WORKLOADS[name])
            oin = di.make_prefill_inputs(ow_)
            oq, ok_, ov, owd = (up(oin[x]) for x in ("q", "k", "v", "wd"))
            del oin
            oo = torch.empty_like(oq)
            osh = dar.make_shape(ow_.B, ow_.Hq, ow_.Hkv, ow_.d, ow_.dd, ow_.w, torch.bfloat16)
            ows = torch.empty(max(1, dar.dar_prefill_workspace_bytes(osh, ow_.T)),
                              dtype=torch.uint8, device=dev)
            run = lambda i: dar.dar_attn_prefill(oq, ok_, ov, owd, None, ow_.w, o=oo, ws=ows,
                                                 check=False)
            for i in range(args.warmup):
                run(i)
            oms = timed(run, args.steps)
            ofl = prefill_flops(ow_.B, ow_.Hq, ow_.T, ow_.d, ow_.dd, ow_.w)
            otf = ofl / (oms * 1e-3) / 1e12
            other[name] = {"shape": "B%d Hq%d Hkv%d T%d d%d d_down%d w%d" % (
                               ow_.B, ow_.Hq, ow_.Hkv, ow_.T, ow_.d, ow_.dd, ow_.w),
                           "us": round(oms * 1e3, 2), "tflops": round(otf, 2),
                           "frac_bf16_peak": round(otf / PEAK_BF16_TFLOPS, 4)}
            del oq, ok_, ov, owd, oo, ows

    # ---------------- prefill backward (the training step's attention part),
    # timed on its own after the steps above
    bwd = None
    if not args.no_backward:
        dgrad = up(di.make_backward_inputs(pw)["dout"])
        o_f, lse_f = dar.dar_attn_prefill(q, k, v, wd, None, pw.w, ws=ws, return_lse=True)
        bws = torch.empty(dar.dar_prefill_backward_workspace_bytes(shape, pw.T), dtype=torch.uint8,
                          device=dev)
        for _ in range(args.warmup):
            dar.dar_attn_prefill_backward(q, k, v, wd, None, pw.w, o_f, lse_f, dgrad, ws=bws,
                                          check=False)
        torch.cuda.synchronize()
        bwd_ms = timed(lambda i: dar.dar_attn_prefill_backward(q, k, v, wd, None, pw.w, o_f, lse_f,
                                                               dgrad, ws=bws, check=False),
                       args.steps)
        bflops = backward_flops(pw.B, pw.Hq, pw.T, pw.d, pw.dd, pw.w)
        bwd_us = float(bwd_ms * 1e3)
        btf = bflops / (bwd_us * 1e-6) / 1e12
        bwd = {"us": round(bwd_us, 2), "tflops": round(btf, 2),
               "frac_bf16_peak": round(btf / PEAK_BF16_TFLOPS, 4), "alg_flop": bflops}
        del bws
        if not args.no_rope:
            # the backward with the rotary embedding (full-d distant keys)
            rpb = dar.Rope(ROPE_PREFILL_DIM, ROPE_BASE, n_pos=pw.T, device=dev)
            o_r, lse_r = dar.dar_attn_prefill_rope(q, k, v, wd, None, pw.w, rpb, return_lse=True)
            rbws = torch.empty(dar.dar_prefill_rope_backward_workspace_bytes(shape, pw.T),
                               dtype=torch.uint8, device=dev)
            run_rb = lambda i: dar.dar_attn_prefill_rope_backward(q, k, v, wd, None, pw.w, rpb, o_r,
                                                                  lse_r, dgrad, ws=rbws)
            for i in range(args.warmup):
                run_rb(i)
            rb_us = float(timed(run_rb, args.steps) * 1e3)
            rbf = full_backward_flops(pw.B, pw.Hq, pw.T, pw.d)
            bwd["rope"] = {"shape": "pythia70m batch, rotary dim %d, base %g" % (ROPE_PREFILL_DIM,
                                                                                ROPE_BASE),
                           "us": round(rb_us, 2), "alg_flop": rbf,
                           "tflops": round(rbf / (rb_us * 1e-6) / 1e12, 2),
                           "frac_bf16_peak": round(rbf / (rb_us * 1e-6) / 1e12 / PEAK_BF16_TFLOPS, 4)}
            del rbws, o_r, lse_r

    launch = None
    if not args.no_launch:
        launch = launch_cost(torch, dar, q, k, v, wd, o, ws, shape, pw, args.steps)

    result = {
        "metric": "DAR prefill TFLOP/s + decode KV GB/s, as fraction of MI355X peak, 1 GPU",
        "value": round(tflops, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(total_ms / args.steps, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded N(0,1) tensors of the workload shapes; no dataset)",
        "config": {
            "workload": "prefill pythia70m-shaped B8 H8 T2048 d64 d_down16 w256 + decode "
                        "1B-shaped B32 Hq32 Hkv8 d64 d_down16 w512 L32768",
            "global_batch": pw.B, "seq_len": pw.T, "parallelism": "none (1 GPU)",
        },
        "prefill": {"us": round(pre_us, 2), "tflops": round(tflops, 2),
                    "frac_bf16_peak": round(tflops / PEAK_BF16_TFLOPS, 4), "alg_flop": flops},
        "decode": {"us": round(dec_us, 2), "gbs": round(gbs, 1),
                   "frac_hbm_peak": round(gbs / PEAK_HBM_GBS, 4), "alg_bytes": dbytes,
                   "cache_len": L_last, "step_cache_len": [L_first, L_last],
                   "append_us": round(float(app_ms * 1e3), 2)},
        "roofline": {"kernel": "dar_attn_prefill (latent pre-pass + attention kernel)",
                     "bound": "mfma", "achieved": round(tflops, 2), "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(tflops / PEAK_BF16_TFLOPS, 4),
                     "traffic": measured_traffic("prefill")},
        "roofline_decode": {"kernel": "dar_attn_decode (split-KV kernel; with one workgroup per "
                                      "(batch, KV head) it also finishes the output, else a "
                                      "combine kernel follows)", "bound": "hbm",
                            "achieved": round(gbs, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                            "frac": round(gbs / PEAK_HBM_GBS, 4),
                            "traffic": measured_traffic("decode")},
        "setup_s": round(setup_s, 1),
    }
    # one exponential per causal pair: the distant region's bound, against the
    # exponential rate measured above at its own clock
    n_exp = float(pw.B * pw.Hq * (pw.T * (pw.T + 1) // 2))
    result["prefill"]["score_elems_per_s"] = n_exp / (pre_us * 1e-6)
    result["prefill"]["frac_exp_ceiling"] = round(n_exp / (pre_us * 1e-6) / k0["exp_per_s"], 4)
    result["k0"] = k0
    if cold:
        cu = float(cold["prefill_ms"] * 1e3)
        result["prefill"]["cold_us"] = round(cu, 2)
        result["prefill"]["cold_tflops"] = round(flops / (cu * 1e-6) / 1e12, 2)
        du = float(cold["decode_ms"] * 1e3)
        result["decode"]["cold_us"] = round(du, 2)
        result["decode"]["cold_gbs"] = round(dbytes / (du * 1e-6) / 1e9, 1)
    if paged:
        pu = float(paged["uniform_ms"] * 1e3)
        pb = decode_bytes(dw.B, dw.Hq, dw.Hkv, dw.d, dw.dd, dw.w, paged["uniform_len"])
        rlu = float(paged["ragged_ms"] * 1e3)
        rb = sum(decode_bytes(1, dw.Hq, dw.Hkv, dw.d, dw.dd, dw.w, n) for n in paged["ragged_lens"])
        result["decode_paged"] = {
            "shape": "decode1b batch, 256-token pages, every sequence at %d tokens"
                     % paged["uniform_len"],
            "us": round(pu, 2), "alg_bytes": pb, "gbs": round(pb / (pu * 1e-6) / 1e9, 1),
            "frac_hbm_peak": round(pb / (pu * 1e-6) / 1e9 / PEAK_HBM_GBS, 4)}
        result["decode_ragged"] = {
            "shape": "decode1b batch, 256-token pages, lengths %d..%d (ragged)"
                     % (min(paged["ragged_lens"]), max(paged["ragged_lens"])),
            "us": round(rlu, 2), "alg_bytes": rb, "gbs": round(rb / (rlu * 1e-6) / 1e9, 1),
            "frac_hbm_peak": round(rb / (rlu * 1e-6) / 1e9 / PEAK_HBM_GBS, 4)}
        if "ragged_rope_ms" in paged:
            rru = float(paged["ragged_rope_ms"] * 1e3)
            result["decode_ragged"]["rope_us"] = round(rru, 2)
            result["decode_ragged"]["rope_frac_hbm_peak"] = round(
                rb / (rru * 1e-6) / 1e9 / PEAK_HBM_GBS, 4)
        sku = float(paged["skewed_ms"] * 1e3)
        sb = sum(decode_bytes(1, dw.Hq, dw.Hkv, dw.d, dw.dd, dw.w, n) for n in paged["skewed_lens"])
        result["decode_skewed"] = {
            "shape": "decode1b batch, 256-token pages, one sequence at %d tokens, %d at 600"
                     % (paged["skewed_lens"][0], dw.B - 1),
            "us": round(sku, 2), "alg_bytes": sb, "gbs": round(sb / (sku * 1e-6) / 1e9, 1),
            "frac_hbm_peak": round(sb / (sku * 1e-6) / 1e9 / PEAK_HBM_GBS, 4)}
    if ragged:
        gu = float(ragged["ms"] * 1e3)
        gfl = sum(prefill_flops(1, pw.Hq, n, pw.d, pw.dd, pw.w) for n in ragged["lens"])
        result["prefill_ragged"] = {
            "shape": "pythia70m batch padded to %d, lengths %d..%d (ragged)"
                     % (pw.T, min(ragged["lens"]), max(ragged["lens"])),
            "us": round(gu, 2), "alg_flop": gfl, "tflops": round(gfl / (gu * 1e-6) / 1e12, 2),
            "frac_bf16_peak": round(gfl / (gu * 1e-6) / 1e12 / PEAK_BF16_TFLOPS, 4)}
    if shared:
        su = float(shared["prefill_ms"] * 1e3)
        result["prefill_shared"] = {
            "shape": "pythia70m batch, one shared latent per token",
            "us": round(su, 2), "alg_flop": flops, "tflops": round(flops / (su * 1e-6) / 1e12, 2),
            "frac_bf16_peak": round(flops / (su * 1e-6) / 1e12 / PEAK_BF16_TFLOPS, 4)}
        sdu = float(shared["decode_ms"] * 1e3)
        sb = decode_bytes_shared(dw.B, dw.Hq, dw.Hkv, dw.d, dw.dd, dw.w, shared["decode_len"])
        result["decode_shared"] = {
            "shape": "decode1b batch, one shared latent per token, %d cached tokens"
                     % shared["decode_len"],
            "us": round(sdu, 2), "alg_bytes": sb, "gbs": round(sb / (sdu * 1e-6) / 1e9, 1),
            "frac_hbm_peak": round(sb / (sdu * 1e-6) / 1e9 / PEAK_HBM_GBS, 4),
            "bytes_vs_two_latents": round(sb / decode_bytes(dw.B, dw.Hq, dw.Hkv, dw.d, dw.dd, dw.w,
                                                            shared["decode_len"]), 4)}
    if rope:
        ru = float(rope["prefill_ms"] * 1e3)
        rfl = full_flops(pw.B, pw.Hq, pw.T, pw.d)
        result["prefill_rope"] = {
            "shape": "pythia70m batch, rotary dim %d of %d, base %g" % (ROPE_PREFILL_DIM, pw.d,
                                                                      ROPE_BASE),
            "us": round(ru, 2), "alg_flop": rfl, "tflops": round(rfl / (ru * 1e-6) / 1e12, 2),
            "frac_bf16_peak": round(rfl / (ru * 1e-6) / 1e12 / PEAK_BF16_TFLOPS, 4)}
        rdu = float(rope["decode_ms"] * 1e3)
        result["decode_rope"] = {
            "shape": "decode1b cache, rotary dim %d, base %g" % (ROPE_DECODE_DIM, ROPE_BASE),
            "us": round(rdu, 2), "gbs": round(dbytes / (rdu * 1e-6) / 1e9, 1),
            "frac_hbm_peak": round(dbytes / (rdu * 1e-6) / 1e9 / PEAK_HBM_GBS, 4)}
        b8 = rope["d128_bytes"]
        r8, p8 = float(rope["d128_decode_ms"] * 1e3), float(rope["d128_plain_ms"] * 1e3)
        result["decode_rope_d128"] = {
            "shape": "B8 Hq32 Hkv8 d128 d_down32 w1024, 16384 cached tokens, rotary dim %d, "
                     "base %g" % (ROPE_DECODE_DIM, ROPE_BASE),
            "us": round(r8, 2), "alg_bytes": b8, "gbs": round(b8 / (r8 * 1e-6) / 1e9, 1),
            "frac_hbm_peak": round(b8 / (r8 * 1e-6) / 1e9 / PEAK_HBM_GBS, 4),
            "plain_decode_us": round(p8, 2),
            "plain_frac_hbm_peak": round(b8 / (p8 * 1e-6) / 1e9 / PEAK_HBM_GBS, 4)}
    if other:
        result["prefill_other"] = other
    if chunk is not None:
        result["prefill_chunk"] = chunk
    if launch is not None:
        result["launch"] = launch
    if bwd is not None:
        result["backward"] = bwd
        result["roofline_backward"] = {
            "kernel": "dar_attn_prefill_backward (preparation, distant and window kernels for "
                      "dq and for dk/dv, weight-share reduction)", "bound": "mfma",
            "achieved": bwd["tflops"], "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
            "frac": bwd["frac_bf16_peak"], "traffic": measured_traffic("backward")}

    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(pw, pin, args.cpu_seconds)

    print(json.dumps(result), flush=True)


def launch_cost(torch, dar, q, k, v, wd, o, ws, shape, pw, n):
    """Host cost of one prefill call and the GPU time of a graph replay.
    host_us_binding: the Python binding (argument checks off) per call;
    host_us_c_abi: the bare C ABI call (ctypes, arguments prepared once):
    validation and two kernel launches; both measured with the GPU kept busy
    so no call waits for it. graph_us: GPU time per replay of a HIP graph
    holding one prefill (pre-pass and attention kernel), back to back, beside
    eager_us, the same calls enqueued eagerly."""
    import ctypes

    n = max(n, 20)
    st = torch.cuda.current_stream()
    wsb = ws.numel()
    args_c = (ctypes.byref(shape), pw.T, ctypes.c_void_p(q.data_ptr()), ctypes.c_void_p(k.data_ptr()),
              ctypes.c_void_p(v.data_ptr()), ctypes.c_void_p(wd.data_ptr()), None,
              ctypes.c_void_p(o.data_ptr()), ctypes.c_void_p(ws.data_ptr()), wsb,
              ctypes.c_void_p(st.cuda_stream))
    torch.cuda.synchronize()
    torch.cuda._sleep(int(2.4e9 * 2e-3 * n))
    t0 = time.perf_counter()
    for _ in range(n):
        dar.dar_attn_prefill(q, k, v, wd, None, pw.w, o=o, ws=ws, check=False)
    t1 = time.perf_counter()
    for _ in range(n):
        rc = dar.lib.dar_attn_prefill(*args_c)
    t2 = time.perf_counter()
    assert rc == 0, rc
    torch.cuda.synchronize()
    # one prefill captured into a graph (no memset or allocation inside)
    g = torch.cuda.CUDAGraph()
    cs = torch.cuda.Stream()
    cs.wait_stream(st)
    with torch.cuda.stream(cs):
        dar.dar_attn_prefill(q, k, v, wd, None, pw.w, o=o, ws=ws, check=False)
        torch.cuda.synchronize()
        with torch.cuda.graph(g, stream=cs):
            dar.dar_attn_prefill(q, k, v, wd, None, pw.w, o=o, ws=ws, check=False)
    st.wait_stream(cs)
    torch.cuda.synchronize()

    def gpu_time(fn):
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        torch.cuda._sleep(int(2.4e9 * 1e-3 * n))
        e0.record()
        for _ in range(n):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / n * 1e3

    graph_us = gpu_time(g.replay)
    eager_us = gpu_time(lambda: dar.dar_attn_prefill(q, k, v, wd, None, pw.w, o=o, ws=ws,
                                                     check=False))
    t3 = time.perf_counter()
    for _ in range(n):
        g.replay()
    t4 = time.perf_counter()
    torch.cuda.synchronize()
    del g
    return {"host_us_binding": round((t1 - t0) / n * 1e6, 2),
            "host_us_c_abi": round((t2 - t1) / n * 1e6, 2),
            "host_us_graph_replay": round((t4 - t3) / n * 1e6, 2),
            "graph_us": round(graph_us, 2), "eager_us": round(eager_us, 2), "calls": n}


def cpu_model():
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(pw, pin, budget_s):
    """The fp64 oracle on the host cores: on whole (batch, head) slices of the
    same prefill workload, cycling over the slices until the time budget is
    used (at least one slice), with every OpenMP thread; then with one thread
    on the tiny workload (whole) and on single pythia70m slices."""
    import dar_inputs as di
    from oracle import oracle

    grp = pw.Hq // pw.Hkv
    pos = np.arange(pw.T)
    per_head = prefill_flops(1, 1, pw.T, pw.d, pw.dd, pw.w)
    n_slices = pw.B * pw.Hq
    threads = oracle.num_threads()
    done = 0
    t0 = time.time()
    while done == 0 or time.time() - t0 < budget_s:
        b, h = divmod(done % n_slices, pw.Hq)
        g = h // grp
        oracle.rows(pin["k"].f64[b, g], pin["v"].f64[b, g], pin["wd"].f64[g], None, pw.w, pos,
                    pin["q"].f64[b, h])
        done += 1
    el = time.time() - t0
    out = {"value": round(done * per_head / el / 1e12, 6), "unit": "TFLOP/s",
           "cores": threads, "kind": "oracle", "cpu_model": cpu_model(),
           "sample": "%d (batch, head) slices (cycling over the %d of the pythia70m prefill), "
                     "all %d rows each, %.1f s, %d threads" % (done, n_slices, pw.T, el, threads)}

    # one thread (the oracle's OpenMP count is left at 1 afterwards: this runs last)
    def one_thread(inp, wl, budget):
        sl = lambda t: t.f64[0:1, 0:1]
        fl = prefill_flops(1, 1, wl.T, wl.d, wl.dd, wl.w)
        n = 0
        t1 = time.time()
        while n == 0 or time.time() - t1 < budget:
            oracle.prefill(sl(inp["q"]), sl(inp["k"]), sl(inp["v"]), inp["wd"].f64[0:1], None, wl.w,
                           threads=1)
            n += 1
        e = time.time() - t1
        return {"value": round(n * fl / e / 1e12, 6), "unit": "TFLOP/s", "cores": 1,
                "sample": "%d prefills of one (batch, head) slice, %.2f s" % (n, e)}

    tw = di.WORKLOADS["tiny"]
    out["single_thread"] = {"tiny": one_thread(di.make_prefill_inputs(tw), tw, 0.5),
                            "pythia70m": one_thread(pin, pw, 3.0)}
    return out


def copy_calibration(torch, dev, nbytes=1 << 28, reps=5):
    """A plain device-to-device copy of known size. Under a hardware-counter
    profile its FETCH_SIZE / WRITE_SIZE per dispatch, against nbytes, gives
    the factor that turns those counters into HBM bytes."""
    src = torch.empty(nbytes // 4, dtype=torch.int32, device=dev).fill_(1)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration": {"bytes_read": nbytes, "bytes_written": nbytes,
                                           "dispatches": reps}}), flush=True)


if __name__ == "__main__":
    main()
