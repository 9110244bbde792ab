"""Python entry to the fp64 DAR oracle (oracle/dar_oracle.c).

TEST INFRASTRUCTURE ONLY: imported by tests, the smoke check and the
benchmark's CPU-baseline leg. The product package never imports this module.

Functions follow the paper's method section:
  down()      Eq. 1, c = x W_down
  lift()      Eq. 1 then Eq. 2, x' = (x W_down) W_up
  rows()      Eq. 3-4 for chosen query rows of one head
  prefill()   Eq. 3-4 for every row of a batch (causal prefill); optionally
              the log of each row's softmax denominator
  backward()  gradients of sum(dO * O) of the prefill (Section 2.3, the
              training setting) with respect to Q, K, V, W_down, W_up
  rope()      the rotary position embedding of Eq. 3 (rotate-half pairing)
  rope_table()   its cos/sin per position and pair
  rows_rope(), prefill_rope()   Eq. 3-4 with RoPE where Eq. 3 applies it:
              on the window key, and on the distant key after the lift
  rows_shared(), prefill_shared()   Eq. 3-4 with one shared latent per token
              (distant key c U_K, distant value c U_V; the Limitations
              section's h^D cache)
  cache_model()  where the split cache keeps each token after n appends
                 (the efficient cache of the Limitations section: full K/V for
                 the last w tokens, the d_down latent for older ones)
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(_HERE, "dar_oracle.c")
LIB = os.path.join(_HERE, "libdar_oracle.so")

_dp = ctypes.POINTER(ctypes.c_double)
_ip = ctypes.POINTER(ctypes.c_int)

GCC_FLAGS = ["-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared", "-fno-fast-math",
             "-ffp-contract=off"]


def compile_source(src: str, out: str) -> str:
    """Compile an oracle C source into a shared library (strict IEEE fp64)."""
    tmp = out + ".tmp%d" % os.getpid()
    subprocess.check_call(["gcc", *GCC_FLAGS, src, "-o", tmp, "-lm"])
    os.replace(tmp, out)
    return out


def build(force: bool = False) -> str:
    if force or not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
        compile_source(SRC, LIB)
    return LIB


def _c64(a):
    return np.ascontiguousarray(a, dtype=np.float64)


def _ptr(a):
    return None if a is None else a.ctypes.data_as(_dp)


class Oracle:
    """Bindings to one build of the oracle library."""

    def __init__(self, path: str):
        lib = ctypes.CDLL(path)
        lib.dar_oracle_rows.restype = ctypes.c_int
        lib.dar_oracle_rows.argtypes = [ctypes.c_int] * 4 + [_dp, _dp, _dp, _dp, ctypes.c_int,
                                                             _ip, _dp, _dp, _dp, _dp]
        lib.dar_oracle_prefill.restype = ctypes.c_int
        lib.dar_oracle_prefill.argtypes = [ctypes.c_int] * 7 + [_dp] * 7 + [ctypes.c_int]
        lib.dar_oracle_down.restype = None
        lib.dar_oracle_down.argtypes = [ctypes.c_int] * 3 + [_dp, _dp, _dp]
        lib.dar_oracle_up.restype = None
        lib.dar_oracle_up.argtypes = [ctypes.c_int] * 3 + [_dp, _dp, _dp, _dp]
        lib.dar_oracle_num_threads.restype = ctypes.c_int
        lib.dar_oracle_rope.restype = None
        lib.dar_oracle_rope.argtypes = [ctypes.c_int] * 3 + [ctypes.c_double, _ip, _dp, _dp]
        lib.dar_oracle_rope_table.restype = None
        lib.dar_oracle_rope_table.argtypes = [ctypes.c_int, ctypes.c_double, ctypes.c_int, _dp]
        lib.dar_oracle_rows_rope.restype = ctypes.c_int
        lib.dar_oracle_rows_rope.argtypes = ([ctypes.c_int] * 5 + [ctypes.c_double, ctypes.c_int]
                                             + [_dp] * 4 + [ctypes.c_int, _ip, _dp, _dp, _dp])
        lib.dar_oracle_prefill_rope.restype = ctypes.c_int
        lib.dar_oracle_prefill_rope.argtypes = ([ctypes.c_int] * 8 + [ctypes.c_double, ctypes.c_int]
                                                + [_dp] * 7 + [ctypes.c_int])
        lib.dar_oracle_rows_shared.restype = ctypes.c_int
        lib.dar_oracle_rows_shared.argtypes = ([ctypes.c_int] * 4 + [_dp] * 5
                                               + [ctypes.c_int, _ip, _dp, _dp, _dp])
        lib.dar_oracle_prefill_shared.restype = ctypes.c_int
        lib.dar_oracle_prefill_shared.argtypes = [ctypes.c_int] * 7 + [_dp] * 8 + [ctypes.c_int]
        lib.dar_oracle_backward.restype = ctypes.c_int
        lib.dar_oracle_backward.argtypes = [ctypes.c_int] * 7 + [_dp] * 11 + [ctypes.c_int]
        lib.dar_oracle_backward_rope.restype = ctypes.c_int
        lib.dar_oracle_backward_rope.argtypes = ([ctypes.c_int] * 8 + [ctypes.c_double, ctypes.c_int]
                                                 + [_dp] * 11 + [ctypes.c_int])
        self.lib = lib

    def num_threads(self) -> int:
        return self.lib.dar_oracle_num_threads()

    def down(self, x, wd):
        """Eq. 1 for every row of x [n, d] with wd [d, dd]."""
        x = _c64(x)
        wd = _c64(wd)
        n, d = x.shape
        dd = wd.shape[1]
        out = np.empty((n, dd), np.float64)
        self.lib.dar_oracle_down(n, d, dd, _ptr(x), _ptr(wd), _ptr(out))
        return out

    def lift(self, x, wd, wu=None):
        """Eq. 1 then Eq. 2: (x wd) wu, with wu = wd^T when wu is None."""
        x = _c64(x)
        wd = _c64(wd)
        n, d = x.shape
        dd = wd.shape[1]
        h = self.down(x, wd)
        out = np.empty((n, d), np.float64)
        wu_c = None if wu is None else _c64(wu)
        self.lib.dar_oracle_up(n, d, dd, _ptr(h), _ptr(wd), _ptr(wu_c), _ptr(out))
        return out

    def rows(self, k, v, wd, wu, w, pos, qr, want_p=False):
        """Eq. 3-4 for query vectors qr [n, d] at positions pos, against one
        head's keys/values k, v [T, d]. Returns o [n, d] (and p [n, T])."""
        k = _c64(k)
        v = _c64(v)
        wd = _c64(wd)
        wu_c = None if wu is None else _c64(wu)
        qr = _c64(qr)
        T, d = k.shape
        dd = wd.shape[1]
        pos = np.ascontiguousarray(pos, dtype=np.int32)
        n = pos.shape[0]
        o = np.empty((n, d), np.float64)
        p = np.empty((n, T), np.float64) if want_p else None
        rc = self.lib.dar_oracle_rows(T, d, dd, int(w), _ptr(k), _ptr(v), _ptr(wd), _ptr(wu_c),
                                      n, pos.ctypes.data_as(_ip), _ptr(qr), _ptr(o), _ptr(p),
                                      None)
        if rc != 0:
            raise ValueError("dar_oracle_rows rejected its arguments")
        return (o, p) if want_p else o

    def prefill(self, q, k, v, wd, wu, w, threads=0, want_lse=False):
        """Causal prefill: q [B,Hq,T,d], k/v [B,Hkv,T,d], wd [Hkv,d,dd], wu [Hkv,dd,d]|None.
        With want_lse also returns lse [B,Hq,T] = log sum_j exp(S_ij), the log of
        each row's softmax denominator (Eq. 4)."""
        q = _c64(q)
        k = _c64(k)
        v = _c64(v)
        wd = _c64(wd)
        wu_c = None if wu is None else _c64(wu)
        B, Hq, T, d = q.shape
        Hkv = k.shape[1]
        dd = wd.shape[2]
        o = np.empty_like(q)
        lse = np.empty((B, Hq, T), np.float64) if want_lse else None
        rc = self.lib.dar_oracle_prefill(B, Hq, Hkv, T, d, dd, int(w), _ptr(q), _ptr(k),
                                         _ptr(v), _ptr(wd), _ptr(wu_c), _ptr(o), _ptr(lse),
                                         int(threads))
        if rc != 0:
            raise ValueError("dar_oracle_prefill rejected its arguments")
        return (o, lse) if want_lse else o

    def rope(self, x, pos, r, base):
        """RoPE of each row x [n, d] at positions pos [n] (Eq. 3)."""
        x = _c64(x)
        n, d = x.shape
        pos = np.ascontiguousarray(pos, dtype=np.int32)
        assert pos.shape == (n,) and 0 <= r <= d and r % 2 == 0
        out = np.empty_like(x)
        self.lib.dar_oracle_rope(n, d, int(r), float(base), pos.ctypes.data_as(_ip), _ptr(x),
                                 _ptr(out))
        return out

    def rope_table(self, r, base, n_pos):
        """[n_pos, r]: cos of the r/2 angles of each position, then their sin."""
        tab = np.empty((n_pos, r), np.float64)
        self.lib.dar_oracle_rope_table(int(r), float(base), int(n_pos), _ptr(tab))
        return tab

    def rows_rope(self, k, v, wd, wu, w, r, base, pos0, pos, qr):
        """Eq. 3-4 with RoPE for query vectors qr [n, d] (un-rotated) at row
        indices pos of one head whose tokens k, v [T, d] (un-rotated) sit at
        positions pos0 .. pos0+T-1."""
        k = _c64(k)
        v = _c64(v)
        wd = _c64(wd)
        wu_c = None if wu is None else _c64(wu)
        qr = _c64(qr)
        T, d = k.shape
        dd = wd.shape[1]
        pos = np.ascontiguousarray(pos, dtype=np.int32)
        n = pos.shape[0]
        o = np.empty((n, d), np.float64)
        rc = self.lib.dar_oracle_rows_rope(T, d, dd, int(w), int(r), float(base), int(pos0),
                                           _ptr(k), _ptr(v), _ptr(wd), _ptr(wu_c), n,
                                           pos.ctypes.data_as(_ip), _ptr(qr), _ptr(o), None)
        if rc != 0:
            raise ValueError("dar_oracle_rows_rope rejected its arguments")
        return o

    def prefill_rope(self, q, k, v, wd, wu, w, r, base, pos0=0, threads=0, want_lse=False):
        """Causal prefill with RoPE inside Eq. 3 over positions pos0..pos0+T-1
        (q, k, v un-rotated; shapes as for prefill)."""
        q = _c64(q)
        k = _c64(k)
        v = _c64(v)
        wd = _c64(wd)
        wu_c = None if wu is None else _c64(wu)
        B, Hq, T, d = q.shape
        Hkv = k.shape[1]
        dd = wd.shape[2]
        o = np.empty_like(q)
        lse = np.empty((B, Hq, T), np.float64) if want_lse else None
        rc = self.lib.dar_oracle_prefill_rope(B, Hq, Hkv, T, d, dd, int(w), int(r), float(base),
                                              int(pos0), _ptr(q), _ptr(k), _ptr(v), _ptr(wd),
                                              _ptr(wu_c), _ptr(o), _ptr(lse), int(threads))
        if rc != 0:
            raise ValueError("dar_oracle_prefill_rope rejected its arguments")
        return (o, lse) if want_lse else o

    def rows_shared(self, k, v, c, uk, uv, w, pos, qr):
        """Eq. 3-4 with a shared latent for query vectors qr [n, d] at positions
        pos: window keys/values k, v [T, d], distant key c U_K and value c U_V
        (c [T, dd], uk, uv [dd, d])."""
        k, v, c, uk, uv, qr = (_c64(x) for x in (k, v, c, uk, uv, qr))
        T, d = k.shape
        dd = c.shape[1]
        pos = np.ascontiguousarray(pos, dtype=np.int32)
        n = pos.shape[0]
        o = np.empty((n, d), np.float64)
        rc = self.lib.dar_oracle_rows_shared(T, d, dd, int(w), _ptr(k), _ptr(v), _ptr(c), _ptr(uk),
                                             _ptr(uv), n, pos.ctypes.data_as(_ip), _ptr(qr),
                                             _ptr(o), None)
        if rc != 0:
            raise ValueError("dar_oracle_rows_shared rejected its arguments")
        return o

    def prefill_shared(self, q, k, v, c, uk, uv, w, threads=0, want_lse=False):
        """Causal prefill with the shared latent: c [B,Hkv,T,dd], uk, uv [Hkv,dd,d]."""
        q, k, v, c, uk, uv = (_c64(x) for x in (q, k, v, c, uk, uv))
        B, Hq, T, d = q.shape
        Hkv = k.shape[1]
        dd = c.shape[3]
        o = np.empty_like(q)
        lse = np.empty((B, Hq, T), np.float64) if want_lse else None
        rc = self.lib.dar_oracle_prefill_shared(B, Hq, Hkv, T, d, dd, int(w), _ptr(q), _ptr(k),
                                                _ptr(v), _ptr(c), _ptr(uk), _ptr(uv), _ptr(o),
                                                _ptr(lse), int(threads))
        if rc != 0:
            raise ValueError("dar_oracle_prefill_shared rejected its arguments")
        return (o, lse) if want_lse else o

    def backward(self, q, k, v, wd, wu, w, dout, threads=0):
        """Gradients of sum(dout * O) of the causal prefill (Section 2.3's
        training setting): returns dq, dk, dv, dwd, dwu (dwu is None when
        tied; dwd then holds the gradient of the tied matrix)."""
        q = _c64(q)
        k = _c64(k)
        v = _c64(v)
        wd = _c64(wd)
        wu_c = None if wu is None else _c64(wu)
        dout = _c64(dout)
        B, Hq, T, d = q.shape
        Hkv = k.shape[1]
        dd = wd.shape[2]
        dq = np.empty_like(q)
        dk = np.empty_like(k)
        dv = np.empty_like(v)
        dwd = np.empty_like(wd)
        dwu = None if wu is None else np.empty_like(wu_c)
        rc = self.lib.dar_oracle_backward(B, Hq, Hkv, T, d, dd, int(w), _ptr(q), _ptr(k), _ptr(v),
                                          _ptr(wd), _ptr(wu_c), _ptr(dout), _ptr(dq), _ptr(dk),
                                          _ptr(dv), _ptr(dwd), _ptr(dwu), int(threads))
        if rc != 0:
            raise ValueError("dar_oracle_backward rejected its arguments")
        return dq, dk, dv, dwd, dwu

    def backward_rope(self, q, k, v, wd, wu, w, r, base, dout, pos0=0, threads=0):
        """Gradients of sum(dout * O) of the causal prefill with RoPE inside
        Eq. 3 (q, k, v un-rotated, tokens at positions pos0..pos0+T-1):
        returns dq, dk, dv, dwd, dwu as backward does."""
        q = _c64(q)
        k = _c64(k)
        v = _c64(v)
        wd = _c64(wd)
        wu_c = None if wu is None else _c64(wu)
        dout = _c64(dout)
        B, Hq, T, d = q.shape
        Hkv = k.shape[1]
        dd = wd.shape[2]
        dq = np.empty_like(q)
        dk = np.empty_like(k)
        dv = np.empty_like(v)
        dwd = np.empty_like(wd)
        dwu = None if wu is None else np.empty_like(wu_c)
        rc = self.lib.dar_oracle_backward_rope(B, Hq, Hkv, T, d, dd, int(w), int(r), float(base),
                                               int(pos0), _ptr(q), _ptr(k), _ptr(v), _ptr(wd),
                                               _ptr(wu_c), _ptr(dout), _ptr(dq), _ptr(dk), _ptr(dv),
                                               _ptr(dwd), _ptr(dwu), int(threads))
        if rc != 0:
            raise ValueError("dar_oracle_backward_rope rejected its arguments")
        return dq, dk, dv, dwd, dwu


_default = None


def default() -> Oracle:
    global _default
    if _default is None:
        _default = Oracle(build())
    return _default


def num_threads():
    return default().num_threads()


def down(x, wd):
    return default().down(x, wd)


def lift(x, wd, wu=None):
    return default().lift(x, wd, wu)


def rows(k, v, wd, wu, w, pos, qr, want_p=False):
    return default().rows(k, v, wd, wu, w, pos, qr, want_p)


def prefill(q, k, v, wd, wu, w, threads=0, want_lse=False):
    return default().prefill(q, k, v, wd, wu, w, threads, want_lse)


def backward(q, k, v, wd, wu, w, dout, threads=0):
    return default().backward(q, k, v, wd, wu, w, dout, threads)


def backward_rope(q, k, v, wd, wu, w, r, base, dout, pos0=0, threads=0):
    return default().backward_rope(q, k, v, wd, wu, w, r, base, dout, pos0, threads)


def rope(x, pos, r, base):
    return default().rope(x, pos, r, base)


def rows_shared(k, v, c, uk, uv, w, pos, qr):
    return default().rows_shared(k, v, c, uk, uv, w, pos, qr)


def prefill_shared(q, k, v, c, uk, uv, w, threads=0, want_lse=False):
    return default().prefill_shared(q, k, v, c, uk, uv, w, threads, want_lse)


def rope_table(r, base, n_pos):
    return default().rope_table(r, base, n_pos)


def rows_rope(k, v, wd, wu, w, r, base, pos0, pos, qr):
    return default().rows_rope(k, v, wd, wu, w, r, base, pos0, pos, qr)


def prefill_rope(q, k, v, wd, wu, w, r, base, pos0=0, threads=0, want_lse=False):
    return default().prefill_rope(q, k, v, wd, wu, w, r, base, pos0, threads, want_lse)


def cache_model(n_tokens: int, w: int, cap: int):
    """Where the split cache holds each token after n_tokens appends.

    Returns (ring_pos, lat_valid): ring_pos[s] is the position held by ring
    slot s (or -1 if the slot was never written); lat_valid[e] says whether
    latent slot e holds token e. The window keeps the last w tokens at full
    dimension; a token leaves the window (and is kept as its latent) once w
    newer tokens exist, so token e is a latent iff e < n_tokens - w.
    """
    ring_pos = np.full(max(w, 0), -1, np.int64)
    for p in range(max(0, n_tokens - w), n_tokens):
        ring_pos[p % w] = p
    lat_valid = np.zeros(cap, bool)
    lat_valid[: max(0, n_tokens - w)] = True
    return ring_pos, lat_valid
