"""Pins of the fp64 oracle to things other than itself.

Each check takes an oracle object (oracle.oracle.Oracle) so the same checks
can be run against deliberately broken builds of the oracle source
(tests/test_oracle_mutants.py) to show that they catch plausible mistakes.

References for what is pinned:
  * w >= T: every token is inside the window, Eq. 3 never takes the lifted
    branch, so Eq. 4 is ordinary causal softmax attention (the paper's
    "Vanilla" baseline of Table 1).
  * d_down = d with identity projections: the lifted token equals the token
    (the no-bottleneck setting of Table 4).
  * w = 0: every token, including the query's own, takes the lifted branch;
    the paper's "Uniform reduction" baseline (Table 3's w=0 row equals
    Table 1's uniform d_down=128 row).
  * General w: Eq. 3 over the training-time dual store (both forms kept per
    token, Section 2.3) is a masked softmax attention over 2T keys, computed
    here with the library routine torch.nn.functional.scaled_dot_product_attention.
  * Hand-derived closed forms (tests/golden/hand_examples.json).
  * Pure-Python brute force (oracle/brute.py) on tiny inputs.
"""
from __future__ import annotations

import json
import math
import os

import numpy as np
import torch

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "hand_examples.json")


def rng(seed):
    return np.random.Generator(np.random.PCG64(seed))


def rand_case(seed, B=2, Hq=4, Hkv=2, T=23, d=8, dd=3, untied=True):
    g = rng(seed)
    q = g.standard_normal((B, Hq, T, d))
    k = g.standard_normal((B, Hkv, T, d))
    v = g.standard_normal((B, Hkv, T, d))
    wd = g.standard_normal((Hkv, d, dd)) / math.sqrt(d)
    wu = g.standard_normal((Hkv, dd, d)) / math.sqrt(dd) if untied else None
    return q, k, v, wd, wu


def sdpa(q, k, v, mask=None, causal=False):
    """Library softmax attention in fp64 on the CPU, scale 1/sqrt(d)."""
    tq = torch.from_numpy(np.ascontiguousarray(q, dtype=np.float64))
    tk = torch.from_numpy(np.ascontiguousarray(k, dtype=np.float64))
    tv = torch.from_numpy(np.ascontiguousarray(v, dtype=np.float64))
    m = None if mask is None else torch.from_numpy(mask)
    out = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, attn_mask=m,
                                                           is_causal=causal)
    return out.numpy()


def expand_kv(x, Hq):
    """[B,Hkv,T,d] -> [B,Hq,T,d] with contiguous query-head groups."""
    grp = Hq // x.shape[1]
    return np.repeat(x, grp, axis=1)


def lifted(x, wd, wu):
    """Lift every token with numpy matmuls (independent of the oracle's loops)."""
    wu_full = np.swapaxes(wd, 1, 2) if wu is None else wu
    return np.einsum("bgtd,gde,gef->bgtf", x, wd, wu_full)


def dual_store_reference(q, k, v, wd, wu, w):
    """Eq. 3-4 as a masked SDPA over [lifted tokens ; full tokens] (2T keys)."""
    B, Hq, T, d = q.shape
    kl = lifted(k, wd, wu)
    vl = lifted(v, wd, wu)
    K2 = np.concatenate([expand_kv(kl, Hq), expand_kv(k, Hq)], axis=2)
    V2 = np.concatenate([expand_kv(vl, Hq), expand_kv(v, Hq)], axis=2)
    i = np.arange(T)[:, None]
    j = np.arange(T)[None, :]
    causal = j <= i
    near = (i - j) < w
    mask = np.concatenate([causal & ~near, causal & near], axis=1)
    return sdpa(q, K2, V2, mask=mask)


# ---------------------------------------------------------------- checks

def check_vanilla_when_window_covers(orc, seed=1):
    q, k, v, wd, wu = rand_case(seed)
    T = q.shape[2]
    ref = sdpa(q, expand_kv(k, q.shape[1]), expand_kv(v, q.shape[1]), causal=True)
    for w in (T, T + 7, 10 ** 6):
        o = orc.prefill(q, k, v, wd, wu, w)
        np.testing.assert_allclose(o, ref, rtol=0, atol=1e-12)


def check_rows_inside_window_are_vanilla(orc, seed=2):
    q, k, v, wd, wu = rand_case(seed)
    Hq, T = q.shape[1], q.shape[2]
    ref = sdpa(q, expand_kv(k, Hq), expand_kv(v, Hq), causal=True)
    for w in (1, 5, 11):
        o = orc.prefill(q, k, v, wd, wu, w)
        np.testing.assert_allclose(o[:, :, :w], ref[:, :, :w], rtol=0, atol=1e-12)
        # and beyond the window the bottleneck must change the output
        assert np.max(np.abs(o[:, :, w:] - ref[:, :, w:])) > 1e-3


def check_identity_bottleneck_is_vanilla(orc, seed=3):
    B, Hq, Hkv, T, d = 1, 4, 2, 19, 6
    g = rng(seed)
    q = g.standard_normal((B, Hq, T, d))
    k = g.standard_normal((B, Hkv, T, d))
    v = g.standard_normal((B, Hkv, T, d))
    ref = sdpa(q, expand_kv(k, Hq), expand_kv(v, Hq), causal=True)
    eye = np.stack([np.eye(d)] * Hkv)
    for w in (0, 1, 4):
        o = orc.prefill(q, k, v, eye, eye, w)
        np.testing.assert_allclose(o, ref, rtol=0, atol=1e-12)
    # any orthogonal square W_down with tied W_up is an identity lift
    orth = np.stack([np.linalg.qr(g.standard_normal((d, d)))[0] for _ in range(Hkv)])
    for w in (0, 3):
        o = orc.prefill(q, k, v, orth, None, w)
        np.testing.assert_allclose(o, ref, rtol=0, atol=1e-12)


def check_window_zero_is_uniform_reduction(orc, seed=4):
    for untied in (False, True):
        q, k, v, wd, wu = rand_case(seed, untied=untied)
        Hq = q.shape[1]
        ref = sdpa(q, expand_kv(lifted(k, wd, wu), Hq), expand_kv(lifted(v, wd, wu), Hq),
                   causal=True)
        o = orc.prefill(q, k, v, wd, wu, 0)
        np.testing.assert_allclose(o, ref, rtol=0, atol=1e-12)


def check_dual_store_masked_attention(orc, seed=5):
    for untied in (False, True):
        for w in (1, 2, 4, 9, 22):
            q, k, v, wd, wu = rand_case(seed + w, untied=untied)
            o = orc.prefill(q, k, v, wd, wu, w)
            np.testing.assert_allclose(o, dual_store_reference(q, k, v, wd, wu, w), rtol=0,
                                       atol=1e-12)


def check_softmax_weights(orc, seed=6):
    q, k, v, wd, wu = rand_case(seed, B=1, Hq=1, Hkv=1, T=31)
    T = q.shape[2]
    pos = np.arange(T)
    for w in (0, 1, 7, 40):
        o, p = orc.rows(k[0, 0], v[0, 0], wd[0], wu[0], w, pos, q[0, 0], want_p=True)
        assert np.all(p >= 0)
        np.testing.assert_allclose(p.sum(axis=1), 1.0, rtol=0, atol=1e-13)
        assert np.all(p[np.triu_indices(T, 1)] == 0.0)
        # o is the p-weighted sum of the distance-selected values
        vl = lifted(v, wd, wu)[0, 0]
        sel = np.where((pos[:, None] - pos[None, :]) < w, 1.0, 0.0)
        ref = (p * sel) @ v[0, 0] + (p * (1 - sel)) @ vl
        np.testing.assert_allclose(o, ref, rtol=0, atol=1e-12)


def check_golden(orc):
    with open(GOLDEN) as f:
        cases = json.load(f)["cases"]
    for c in cases:
        q = np.array(c["q"])[None, None]
        k = np.array(c["k"])[None, None]
        v = np.array(c["v"])[None, None]
        wd = np.array(c["wd"])[None]
        wu = None if c["wu"] is None else np.array(c["wu"])[None]
        o = orc.prefill(q, k, v, wd, wu, c["w"])[0, 0]
        np.testing.assert_allclose(o, np.array(c["o"]), rtol=0, atol=1e-12, err_msg=c["name"])


def check_brute_force(orc, seed=7):
    from oracle import brute
    for (B, Hq, Hkv, T, d, dd) in ((1, 2, 1, 9, 4, 2), (2, 2, 2, 6, 3, 1)):
        for untied in (False, True):
            for w in (0, 1, 3, T, T + 2):
                q, k, v, wd, wu = rand_case(seed + w, B, Hq, Hkv, T, d, dd, untied)
                ref = np.array(brute.prefill(q.tolist(), k.tolist(), v.tolist(), wd.tolist(),
                                             None if wu is None else wu.tolist(), w))
                o = orc.prefill(q, k, v, wd, wu, w)
                np.testing.assert_allclose(o, ref, rtol=0, atol=1e-12)


def check_absorption_algebra(orc, seed=8):
    """(q W_up^T).(k W_down) == q.((k W_down) W_up) and (sum p c) W_up == sum p (c W_up):
    the rewrites the efficient cache relies on (Limitations section)."""
    g = rng(seed)
    d, dd, n = 16, 4, 13
    wd = g.standard_normal((d, dd))
    wu = g.standard_normal((dd, d))
    k = g.standard_normal((n, d))
    q = g.standard_normal(d)
    p = g.random(n)
    c = orc.down(k, wd)
    np.testing.assert_allclose(c, k @ wd, rtol=0, atol=1e-12)
    kl = orc.lift(k, wd, wu)
    np.testing.assert_allclose(kl @ q, c @ (wu @ q), rtol=0, atol=1e-12)
    np.testing.assert_allclose(p @ kl, (p @ c) @ wu, rtol=0, atol=1e-12)
    # tied: W_up = W_down^T
    np.testing.assert_allclose(orc.lift(k, wd, None), (k @ wd) @ wd.T, rtol=0, atol=1e-12)


def check_gauge_invariance(orc, seed=9):
    """W_down -> W_down M, W_up -> M^-1 W_up leaves every output unchanged."""
    q, k, v, wd, wu = rand_case(seed, untied=True)
    g = rng(seed + 1)
    M = g.standard_normal((wd.shape[0], wd.shape[2], wd.shape[2])) + 3 * np.eye(wd.shape[2])
    wd2 = np.einsum("gde,gef->gdf", wd, M)
    wu2 = np.einsum("gef,gfd->ged", np.linalg.inv(M), wu)
    for w in (0, 3, 10):
        np.testing.assert_allclose(orc.prefill(q, k, v, wd2, wu2, w),
                                   orc.prefill(q, k, v, wd, wu, w), rtol=0, atol=1e-10)


def check_distant_order_irrelevant(orc, seed=10):
    """Permuting tokens that are all distant for the last row leaves that row alone."""
    q, k, v, wd, wu = rand_case(seed, B=1, Hq=2, Hkv=1, T=30)
    T = q.shape[2]
    for w in (0, 4, 11):
        n_dist = T - w            # positions [0, T-1-w] are distant for row T-1
        perm = np.arange(T)
        perm[:n_dist] = rng(seed + w).permutation(n_dist)
        if w == 0:
            perm[: T - 1] = rng(seed + 99).permutation(T - 1)  # keep the query's own key last
            perm[T - 1] = T - 1
        o1 = orc.prefill(q, k, v, wd, wu, w)[:, :, -1]
        o2 = orc.prefill(q, k[:, :, perm], v[:, :, perm], wd, wu, w)[:, :, -1]
        np.testing.assert_allclose(o1, o2, rtol=0, atol=1e-12)


def check_first_row(orc, seed=11):
    q, k, v, wd, wu = rand_case(seed)
    Hq = q.shape[1]
    vl = lifted(v, wd, wu)
    for w in (0, 1, 5):
        o = orc.prefill(q, k, v, wd, wu, w)
        expect = expand_kv(v if w >= 1 else vl, Hq)[:, :, 0]
        np.testing.assert_allclose(o[:, :, 0], expect, rtol=0, atol=1e-14)


def check_gqa_is_repeated_mha(orc, seed=12):
    q, k, v, wd, wu = rand_case(seed, Hq=6, Hkv=2)
    grp = 3
    wd_rep = np.repeat(wd, grp, axis=0)
    wu_rep = np.repeat(wu, grp, axis=0)
    for w in (0, 5):
        o1 = orc.prefill(q, k, v, wd, wu, w)
        o2 = orc.prefill(q, expand_kv(k, 6), expand_kv(v, 6), wd_rep, wu_rep, w)
        np.testing.assert_allclose(o1, o2, rtol=0, atol=0)


def check_rows_match_prefill(orc, seed=13):
    """The decode-style row entry (arbitrary query vector at a position) agrees
    with the prefill at that position."""
    q, k, v, wd, wu = rand_case(seed, B=1, Hq=1, Hkv=1, T=27)
    pos = np.array([0, 5, 17, 26])
    for w in (0, 6):
        o = orc.rows(k[0, 0], v[0, 0], wd[0], wu[0], w, pos, q[0, 0, pos])
        np.testing.assert_allclose(o, orc.prefill(q, k, v, wd, wu, w)[0, 0, pos], rtol=0,
                                   atol=0)


ALL_CHECKS = [
    check_vanilla_when_window_covers,
    check_rows_inside_window_are_vanilla,
    check_identity_bottleneck_is_vanilla,
    check_window_zero_is_uniform_reduction,
    check_dual_store_masked_attention,
    check_softmax_weights,
    check_golden,
    check_brute_force,
    check_absorption_algebra,
    check_gauge_invariance,
    check_distant_order_irrelevant,
    check_first_row,
    check_gqa_is_repeated_mha,
    check_rows_match_prefill,
]
