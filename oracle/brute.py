"""Scalar brute-force DAR attention, pure Python loops, for tiny inputs only.

TEST INFRASTRUCTURE ONLY. Written independently of dar_oracle.c (different
language, different loop structure: it materialises the distance-selected key
and value rows of Eq. 3 for each query before applying Eq. 4), so that a
mistake in one is unlikely to be repeated in the other.
"""
from __future__ import annotations

import math


def _matvec_rows(x, m):
    """x: list of rows (len n), m: [len(x[0])][cols] -> n x cols."""
    cols = len(m[0])
    return [[sum(xr[e] * m[e][c] for e in range(len(xr))) for c in range(cols)] for xr in x]


def attend_head(q, k, v, wd, wu, w):
    """q, k, v: T x d nested lists; wd: d x dd; wu: dd x d or None (tied)."""
    T = len(q)
    d = len(q[0])
    dd = len(wd[0])
    if wu is None:
        wu = [[wd[e][c] for e in range(d)] for c in range(dd)]
    # Eq. 1 and Eq. 2 for every token
    k_lift = _matvec_rows(_matvec_rows(k, wd), wu)
    v_lift = _matvec_rows(_matvec_rows(v, wd), wu)
    out = []
    for i in range(T):
        # Eq. 3: distance-selected keys and values for query i
        keys = []
        vals = []
        for j in range(i + 1):
            near = (i - j) < w
            keys.append(k[j] if near else k_lift[j])
            vals.append(v[j] if near else v_lift[j])
        # Eq. 4
        logits = [sum(q[i][e] * key[e] for e in range(d)) / math.sqrt(d) for key in keys]
        top = max(logits)
        ex = [math.exp(s - top) for s in logits]
        z = sum(ex)
        out.append([sum(ex[j] / z * vals[j][e] for j in range(len(vals))) for e in range(d)])
    return out


def prefill(q, k, v, wd, wu, w):
    """q [B][Hq][T][d], k/v [B][Hkv][T][d], wd [Hkv][d][dd], wu [Hkv][dd][d] or None."""
    B = len(q)
    Hq = len(q[0])
    Hkv = len(k[0])
    grp = Hq // Hkv
    return [[attend_head(q[b][h], k[b][h // grp], v[b][h // grp], wd[h // grp],
                         None if wu is None else wu[h // grp], w)
             for h in range(Hq)] for b in range(B)]
