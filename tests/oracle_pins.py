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

RoPE inside Eq. 3 (rotate-half pairing, window keys rotated as they are,
distant keys rotated after the lift, values never):
  * the rotation against its complex-number form (each pair as one complex
    number multiplied by exp(i * angle)) and against cos/sin of 1 and 3
    radians written out;
  * r = 0 is the plain prefill;
  * every score depends on positions only through i - j (the defining
    property of rotary embeddings), so shifting all positions leaves the
    output unchanged; a rotation skipped, misplaced or applied before the
    lift breaks this;
  * general w: the dual-store masked attention above with the keys rotated
    in complex form (w >= T: causal attention over rotated queries and keys).

Single shared latent (one d_down vector c_j per token and KV head, distant
key c_j U_K, distant value c_j U_V; the Limitations section's cache):
  * with v = k, c = k W_down and U_K = U_V = W_down^T it is the two-latent
    oracle above (pinned);
  * general w: the dual-store masked attention with keys [c U_K ; k] and
    values [c U_V ; v], written with numpy products and library SDPA;
  * w >= T: causal attention over k, v alone (no latent is read);
  * w = 0: attention over (c U_K, c U_V) alone, the row's own token included.

Backward (gradients of sum(dO * O), the training setting of Section 2.3):
  * central finite differences of the forward prefill (itself pinned above);
  * torch fp64 autograd of the dual-store masked attention, written here with
    plain tensor ops;
  * w >= T: ordinary causal attention's autograd, and exactly zero gradient
    for W_down and W_up, which the paper says are updated only from positions
    whose query takes the global path;
  * closed forms: T = 1, Euler's identity <dV, V> = sum(dO * O) (O is linear
    in V), and the gauge identity W_down^T dW_down = dW_up W_up^T that follows
    from the invariance under W_down -> W_down M, W_up -> M^-1 W_up.
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


def check_log_sum_exp(orc, seed=14):
    """The row log-sum-exp equals torch.logsumexp of the masked dual-store
    scores (library routine), and, with w >= T, of plain causal scores."""
    for untied in (False, True):
        for w in (0, 3, 23, 40):
            q, k, v, wd, wu = rand_case(seed + w, untied=untied)
            _, lse = orc.prefill(q, k, v, wd, wu, w, want_lse=True)
            B, Hq, T, d = q.shape
            kl = lifted(k, wd, wu)
            K2 = np.concatenate([expand_kv(kl, Hq), expand_kv(k, Hq)], axis=2)
            S = torch.from_numpy(np.einsum("bhid,bhjd->bhij", q, K2) / math.sqrt(d))
            i = np.arange(T)[:, None]
            j = np.arange(T)[None, :]
            mask = np.concatenate([(j <= i) & ((i - j) >= w), (j <= i) & ((i - j) < w)], axis=1)
            ref = torch.logsumexp(S.masked_fill(~torch.from_numpy(mask), float("-inf")), dim=-1)
            np.testing.assert_allclose(lse, ref.numpy(), rtol=0, atol=1e-12)


# ---------------------------------------------------------------- backward

def torch_dual_store(q, k, v, wd, wu, w):
    """Eq. 3-4 over the dual store with plain torch ops (differentiable):
    [lifted tokens ; full tokens] as 2T keys, the distance picking one of each
    pair through the mask."""
    B, Hq, T, d = q.shape
    G = Hq // k.shape[1]
    wu_full = wd.transpose(1, 2) if wu is None else wu
    lift = lambda x: torch.matmul(torch.matmul(x, wd[None]), wu_full[None])
    K2 = torch.cat([lift(k), k], dim=2).repeat_interleave(G, dim=1)
    V2 = torch.cat([lift(v), v], dim=2).repeat_interleave(G, dim=1)
    s = torch.matmul(q, K2.transpose(-1, -2)) / math.sqrt(d)
    i = torch.arange(T)[:, None]
    j = torch.arange(T)[None, :]
    causal = j <= i
    near = (i - j) < w
    mask = torch.cat([causal & ~near, causal & near], dim=1)
    s = s.masked_fill(~mask, float("-inf"))
    return torch.matmul(torch.softmax(s, dim=-1), V2)


def torch_grads(fn, dout, *arrays):
    """Gradients of sum(dout * fn(*arrays)) by fp64 autograd on the CPU; a
    None array stays None."""
    ts = [None if a is None else torch.tensor(a, dtype=torch.float64, requires_grad=True)
          for a in arrays]
    out = fn(*ts)
    (out * torch.tensor(dout)).sum().backward()
    return [None if t is None else t.grad.numpy() for t in ts]


def _bwd_case(seed, untied, **kw):
    q, k, v, wd, wu = rand_case(seed, untied=untied, **kw)
    dout = rng(seed + 1000).standard_normal(q.shape)
    return q, k, v, wd, wu, dout


def _assert_grads(got, ref, atol, what):
    names = ("dq", "dk", "dv", "dwd", "dwu")
    for n, a, b in zip(names, got, ref):
        if b is None:
            assert a is None, what + " " + n
            continue
        np.testing.assert_allclose(a, b, rtol=0, atol=atol, err_msg=what + " " + n)


def check_backward_finite_differences(orc, seed=21):
    """Central differences of L = sum(dO * O) through the forward prefill."""
    h = 1e-5
    for untied in (False, True):
        for w in (0, 2, 9):
            q, k, v, wd, wu, dout = _bwd_case(seed + w, untied, B=1, Hq=2, Hkv=1, T=7, d=4,
                                              dd=2)
            got = orc.backward(q, k, v, wd, wu, w, dout)
            args = [q, k, v, wd, wu]
            for a_i, a in enumerate(args):
                if a is None:
                    continue
                fd = np.empty_like(a)
                flat = a.reshape(-1)
                for x in range(flat.size):
                    keep = flat[x]
                    flat[x] = keep + h
                    lp = np.sum(dout * orc.prefill(*args, w))
                    flat[x] = keep - h
                    lm = np.sum(dout * orc.prefill(*args, w))
                    flat[x] = keep
                    fd.reshape(-1)[x] = (lp - lm) / (2 * h)
                np.testing.assert_allclose(got[a_i], fd, rtol=0, atol=1e-7,
                                           err_msg="fd untied=%s w=%d arg %d" % (untied, w, a_i))


def check_backward_dual_store_autograd(orc, seed=22):
    for untied in (False, True):
        for w in (0, 1, 5, 22, 30):
            q, k, v, wd, wu, dout = _bwd_case(seed + w, untied)
            ref = torch_grads(lambda *t: torch_dual_store(*t, w), dout, q, k, v, wd, wu)
            got = orc.backward(q, k, v, wd, wu, w, dout)
            _assert_grads(got, ref, 1e-11, "dual store untied=%s w=%d" % (untied, w))


def check_backward_vanilla_no_bottleneck_gradient(orc, seed=23):
    """w >= T: plain causal attention's gradients; W_down and W_up get none."""
    for untied in (False, True):
        q, k, v, wd, wu, dout = _bwd_case(seed, untied)
        T, Hq = q.shape[2], q.shape[1]

        def vanilla(tq, tk, tv):
            G = Hq // tk.shape[1]
            return torch.nn.functional.scaled_dot_product_attention(
                tq, tk.repeat_interleave(G, dim=1), tv.repeat_interleave(G, dim=1),
                is_causal=True)

        rq, rk, rv = torch_grads(vanilla, dout, q, k, v)
        for w in (T, T + 5):
            dq, dk, dv, dwd, dwu = orc.backward(q, k, v, wd, wu, w, dout)
            _assert_grads((dq, dk, dv), (rq, rk, rv), 1e-12, "vanilla w=%d" % w)
            assert np.all(dwd == 0.0)
            assert dwu is None or np.all(dwu == 0.0)


def check_backward_single_token(orc, seed=24):
    """T = 1: O is the first value (full or lifted), so dq = dk = 0 and the
    value and bottleneck gradients have closed forms."""
    for untied in (False, True):
        q, k, v, wd, wu, dout = _bwd_case(seed, untied, B=2, Hq=4, Hkv=2, T=1, d=6, dd=2)
        dsum = dout.reshape(2, 2, 2, 1, 6).sum(axis=2)      # summed over each head group
        for w in (0, 1, 3):
            dq, dk, dv, dwd, dwu = orc.backward(q, k, v, wd, wu, w, dout)
            assert np.all(dq == 0.0) and np.all(dk == 0.0)
            if w >= 1:
                np.testing.assert_allclose(dv, dsum, rtol=0, atol=1e-14)
                assert np.all(dwd == 0.0)
                continue
            wu_f = np.swapaxes(wd, 1, 2) if wu is None else wu
            for b in range(2):
                for g in range(2):
                    np.testing.assert_allclose(dv[b, g, 0], dsum[b, g, 0] @ (wd[g] @ wu_f[g]).T,
                                               rtol=0, atol=1e-13)
            u = np.einsum("bge,gce->bgc", dsum[:, :, 0], wu_f)          # dO W_up^T
            gwd = np.einsum("bgd,bgc->gdc", v[:, :, 0], u)
            gwu = np.einsum("bgc,bge->gce", np.einsum("bgd,gdc->bgc", v[:, :, 0], wd),
                            dsum[:, :, 0])
            if wu is None:
                np.testing.assert_allclose(dwd, gwd + np.swapaxes(gwu, 1, 2), rtol=0, atol=1e-13)
            else:
                np.testing.assert_allclose(dwd, gwd, rtol=0, atol=1e-13)
                np.testing.assert_allclose(dwu, gwu, rtol=0, atol=1e-13)


def check_backward_identities(orc, seed=25):
    """<dV, V> = sum(dO * O) (O is homogeneous of degree one in V, through
    both paths), and W_down^T dW_down = dW_up W_up^T (gauge invariance)."""
    for w in (0, 3, 10):
        q, k, v, wd, wu, dout = _bwd_case(seed + w, True)
        dq, dk, dv, dwd, dwu = orc.backward(q, k, v, wd, wu, w, dout)
        L = np.sum(dout * orc.prefill(q, k, v, wd, wu, w))
        assert abs(np.sum(dv * v) - L) < 1e-10 * max(1.0, abs(L))
        lhs = np.einsum("gdc,gde->gce", wd, dwd)
        rhs = np.einsum("gcd,ged->gce", dwu, wu)
        np.testing.assert_allclose(lhs, rhs, rtol=0, atol=1e-10)


# ---------------------------------------------------------------- RoPE

def rope_complex(x, pos, r, base):
    """RoPE in complex form: the pair (x[m], x[m + r/2]) is the complex number
    x[m] + i x[m + r/2], multiplied by exp(i pos base^(-2m/r)); pos broadcasts
    over the rows (second-to-last axis) of x."""
    x = np.asarray(x, np.float64)
    out = x.copy()
    h = r // 2
    if h == 0:
        return out
    ang = np.asarray(pos, np.float64)[:, None] * float(base) ** (-2.0 * np.arange(h) / r)
    z = (x[..., :h] + 1j * x[..., h:r]) * np.exp(1j * ang)
    out[..., :h] = z.real
    out[..., h:r] = z.imag
    return out


def check_rope_rotation(orc, seed=31):
    # cos and sin of 1 and 3 radians: with r = 2 the only angle is the position
    got = orc.rope(np.array([[1.0, 0.0], [0.0, 1.0]]), [1, 3], 2, 10000.0)
    want = np.array([[0.5403023058681398, 0.8414709848078965],
                     [-0.1411200080598672, -0.9899924966004454]])
    np.testing.assert_allclose(got, want, rtol=0, atol=1e-15)
    g = rng(seed)
    for d, r, base in ((8, 8, 10000.0), (8, 4, 10000.0), (12, 6, 500000.0), (6, 0, 10.0)):
        x = g.standard_normal((40, d))
        pos = g.integers(0, 40000, 40)
        np.testing.assert_allclose(orc.rope(x, pos, r, base), rope_complex(x, pos, r, base),
                                   rtol=0, atol=1e-9)
        if r:
            ang = np.arange(50)[:, None] * base ** (-2.0 * np.arange(r // 2) / r)
            tab = orc.rope_table(r, base, 50)
            np.testing.assert_allclose(tab[:, : r // 2], np.exp(1j * ang).real, rtol=0, atol=1e-12)
            np.testing.assert_allclose(tab[:, r // 2:], np.exp(1j * ang).imag, rtol=0, atol=1e-12)


def check_rope_zero_dim_is_plain(orc, seed=32):
    q, k, v, wd, wu = rand_case(seed)
    for w in (0, 4, 100):
        np.testing.assert_allclose(orc.prefill_rope(q, k, v, wd, wu, w, 0, 10000.0, pos0=9),
                                   orc.prefill(q, k, v, wd, wu, w), rtol=0, atol=1e-15)


def check_rope_shift_invariance(orc, seed=33):
    q, k, v, wd, wu = rand_case(seed, d=8, dd=3)
    for w, r in ((5, 8), (1, 4), (0, 8), (30, 6)):
        a = orc.prefill_rope(q, k, v, wd, wu, w, r, 100.0, pos0=0)
        b = orc.prefill_rope(q, k, v, wd, wu, w, r, 100.0, pos0=1237)
        np.testing.assert_allclose(a, b, rtol=0, atol=1e-10)
    # and the rotation does change the output
    assert np.abs(a - orc.prefill(q, k, v, wd, wu, 30)).max() > 1e-3


def check_rope_dual_store(orc, seed=34):
    q, k, v, wd, wu = rand_case(seed, d=8, dd=3)
    B, Hq, T, d = q.shape
    for w, r, pos0, base in ((5, 6, 3, 50.0), (0, 8, 0, 10000.0), (T, 8, 11, 10.0),
                             (9, 4, 2000, 10000.0)):
        pos = pos0 + np.arange(T)
        kl = lifted(k, wd, wu)
        vl = lifted(v, wd, wu)
        K2 = np.concatenate([expand_kv(rope_complex(kl, pos, r, base), Hq),
                             expand_kv(rope_complex(k, pos, r, base), Hq)], axis=2)
        V2 = np.concatenate([expand_kv(vl, Hq), expand_kv(v, Hq)], axis=2)
        i = np.arange(T)[:, None]
        j = np.arange(T)[None, :]
        causal = j <= i
        near = (i - j) < w
        mask = np.concatenate([causal & ~near, causal & near], axis=1)
        ref = sdpa(rope_complex(q, pos, r, base), K2, V2, mask=mask)
        got = orc.prefill_rope(q, k, v, wd, wu, w, r, base, pos0=pos0)
        np.testing.assert_allclose(got, ref, rtol=0, atol=1e-12)
        # the per-row entry point gives the same rows
        rows = np.array([0, 3, T - 1])
        o = orc.rows_rope(k[1, 0], v[1, 0], wd[0], None if wu is None else wu[0], w, r, base, pos0,
                          rows, q[1, 1, rows])
        np.testing.assert_allclose(o, got[1, 1, rows], rtol=0, atol=1e-12)


def torch_rope_complex(x, pos, r, base):
    """rope_complex in torch (differentiable): the pairs as complex numbers
    multiplied by unit phasors."""
    h = r // 2
    if h == 0:
        return x
    ang = torch.as_tensor(np.asarray(pos, np.float64))[:, None] * float(base) ** (
        -2.0 * torch.arange(h, dtype=torch.float64) / r)
    z = torch.complex(x[..., :h], x[..., h:r]) * torch.polar(torch.ones_like(ang), ang)
    return torch.cat([z.real, z.imag, x[..., r:]], dim=-1)


def torch_dual_store_rope(q, k, v, wd, wu, w, r, base, pos0):
    """Eq. 3-4 with RoPE over the dual store in torch: lifted-then-rotated and
    rotated keys as 2T keys, lifted and plain values, the distance picking one
    of each pair."""
    B, Hq, T, d = q.shape
    G = Hq // k.shape[1]
    pos = pos0 + np.arange(T)
    wu_full = wd.transpose(1, 2) if wu is None else wu
    lift = lambda x: torch.matmul(torch.matmul(x, wd[None]), wu_full[None])
    K2 = torch.cat([torch_rope_complex(lift(k), pos, r, base), torch_rope_complex(k, pos, r, base)],
                   dim=2).repeat_interleave(G, dim=1)
    V2 = torch.cat([lift(v), v], dim=2).repeat_interleave(G, dim=1)
    s = torch.matmul(torch_rope_complex(q, pos, r, base), K2.transpose(-1, -2)) / math.sqrt(d)
    i = torch.arange(T)[:, None]
    j = torch.arange(T)[None, :]
    causal = j <= i
    near = (i - j) < w
    mask = torch.cat([causal & ~near, causal & near], dim=1)
    s = s.masked_fill(~mask, float("-inf"))
    return torch.matmul(torch.softmax(s, dim=-1), V2)


def check_backward_rope_finite_differences(orc, seed=35):
    """Central differences of L = sum(dO * O) through the rotary forward."""
    h = 1e-5
    for untied in (False, True):
        for w, r in ((0, 4), (2, 2), (9, 4)):
            q, k, v, wd, wu, dout = _bwd_case(seed + w, untied, B=1, Hq=2, Hkv=1, T=7, d=4,
                                              dd=2)
            got = orc.backward_rope(q, k, v, wd, wu, w, r, 100.0, dout, pos0=3)
            args = [q, k, v, wd, wu]
            for a_i, a in enumerate(args):
                if a is None:
                    continue
                fd = np.empty_like(a)
                flat = a.reshape(-1)
                for x in range(flat.size):
                    keep = flat[x]
                    flat[x] = keep + h
                    lp = np.sum(dout * orc.prefill_rope(*args, w, r, 100.0, pos0=3))
                    flat[x] = keep - h
                    lm = np.sum(dout * orc.prefill_rope(*args, w, r, 100.0, pos0=3))
                    flat[x] = keep
                    fd.reshape(-1)[x] = (lp - lm) / (2 * h)
                np.testing.assert_allclose(got[a_i], fd, rtol=0, atol=1e-7,
                                           err_msg="rope fd untied=%s w=%d arg %d" % (untied, w, a_i))


def check_backward_rope_dual_store_autograd(orc, seed=36):
    for untied in (False, True):
        for w, r, pos0, base in ((0, 8, 5, 10000.0), (3, 6, 0, 50.0), (9, 4, 700, 10000.0),
                                 (40, 8, 2, 10.0)):
            q, k, v, wd, wu, dout = _bwd_case(seed + w, untied, d=8, dd=3)
            ref = torch_grads(lambda *t: torch_dual_store_rope(*t, w, r, base, pos0), dout,
                              q, k, v, wd, wu)
            got = orc.backward_rope(q, k, v, wd, wu, w, r, base, dout, pos0=pos0)
            _assert_grads(got, ref, 1e-11, "rope dual store untied=%s w=%d r=%d" % (untied, w, r))


def check_backward_rope_zero_dim_is_plain(orc, seed=37):
    for untied in (False, True):
        q, k, v, wd, wu, dout = _bwd_case(seed, untied)
        for w in (0, 4, 100):
            got = orc.backward_rope(q, k, v, wd, wu, w, 0, 10000.0, dout, pos0=9)
            _assert_grads(got, orc.backward(q, k, v, wd, wu, w, dout), 1e-15, "rope r=0 w=%d" % w)


def check_backward_rope_shift_invariance(orc, seed=38):
    """The scores depend on relative positions only, and the gradients of the
    un-rotated inputs are rotated back: shifting every position changes none."""
    q, k, v, wd, wu, dout = _bwd_case(seed, True, d=8, dd=3)
    for w, r in ((5, 8), (0, 6)):
        a = orc.backward_rope(q, k, v, wd, wu, w, r, 100.0, dout, pos0=0)
        b = orc.backward_rope(q, k, v, wd, wu, w, r, 100.0, dout, pos0=1237)
        _assert_grads(b, a, 1e-9, "rope shift w=%d" % w)
    # and the rotation does change the gradients
    assert np.abs(a[0] - orc.backward(q, k, v, wd, wu, 0, dout)[0]).max() > 1e-3


# ---------------------------------------------------------------- shared latent

def shared_case(seed, B=2, Hq=4, Hkv=2, T=23, d=8, dd=3):
    g = rng(seed)
    q = g.standard_normal((B, Hq, T, d))
    k = g.standard_normal((B, Hkv, T, d))
    v = g.standard_normal((B, Hkv, T, d))
    c = g.standard_normal((B, Hkv, T, dd))
    uk = g.standard_normal((Hkv, dd, d)) / math.sqrt(dd)
    uv = g.standard_normal((Hkv, dd, d)) / math.sqrt(dd)
    return q, k, v, c, uk, uv


def check_shared_reduces_to_two_latents(orc, seed=41):
    q, k, v, wd, wu = rand_case(seed, untied=False)
    c = np.einsum("bgtd,gde->bgte", k, wd)
    wdt = np.ascontiguousarray(np.swapaxes(wd, 1, 2))
    for w in (0, 3, 9):
        np.testing.assert_allclose(orc.prefill_shared(q, k, k, c, wdt, wdt, w),
                                   orc.prefill(q, k, k, wd, None, w), rtol=0, atol=1e-12)


def check_shared_dual_store(orc, seed=42):
    q, k, v, c, uk, uv = shared_case(seed)
    B, Hq, T, d = q.shape
    i = np.arange(T)[:, None]
    j = np.arange(T)[None, :]
    for w in (0, 1, 6, T, T + 5):
        kl = np.einsum("bgtc,gcd->bgtd", c, uk)
        vl = np.einsum("bgtc,gcd->bgtd", c, uv)
        K2 = np.concatenate([expand_kv(kl, Hq), expand_kv(k, Hq)], axis=2)
        V2 = np.concatenate([expand_kv(vl, Hq), expand_kv(v, Hq)], axis=2)
        causal = j <= i
        near = (i - j) < w
        mask = np.concatenate([causal & ~near, causal & near], axis=1)
        got = orc.prefill_shared(q, k, v, c, uk, uv, w)
        np.testing.assert_allclose(got, sdpa(q, K2, V2, mask=mask), rtol=0, atol=1e-12)
        if w >= T:   # no latent is read
            ref = sdpa(q, expand_kv(k, Hq), expand_kv(v, Hq), causal=True)
            np.testing.assert_allclose(got, ref, rtol=0, atol=1e-12)
        if w == 0:   # every token through the latent, its own included
            ref = sdpa(q, expand_kv(kl, Hq), expand_kv(vl, Hq), causal=True)
            np.testing.assert_allclose(got, ref, rtol=0, atol=1e-12)
    rows = np.array([0, 5, T - 1])
    o = orc.rows_shared(k[1, 1], v[1, 1], c[1, 1], uk[1], uv[1], 6, rows, q[1, 3, rows])
    np.testing.assert_allclose(o, orc.prefill_shared(q, k, v, c, uk, uv, 6)[1, 3, rows], rtol=0,
                               atol=1e-12)


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
    check_log_sum_exp,
    check_backward_finite_differences,
    check_backward_dual_store_autograd,
    check_backward_vanilla_no_bottleneck_gradient,
    check_backward_single_token,
    check_backward_identities,
    check_rope_rotation,
    check_rope_zero_dim_is_plain,
    check_rope_shift_invariance,
    check_rope_dual_store,
    check_backward_rope_finite_differences,
    check_backward_rope_dual_store_autograd,
    check_backward_rope_zero_dim_is_plain,
    check_backward_rope_shift_invariance,
    check_shared_reduces_to_two_latents,
    check_shared_dual_store,
]
