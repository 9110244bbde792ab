"""DAR attention on MI355X: Python binding of libdar (include/dar.h).

Argument marshalling only: torch provides device memory and the current HIP
stream; every step of the computation runs in the library's HIP kernels.
The library must have been built (paper_2606_18587_amd.build); importing this
package without it raises, there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libdar.so")

DAR_OK, DAR_E_ARG, DAR_E_UNSUPPORTED, DAR_E_CAPACITY, DAR_E_WORKSPACE, DAR_E_HIP = range(6)
DAR_F32, DAR_BF16 = 0, 1


class DarShape(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int), ("Hq", ctypes.c_int), ("Hkv", ctypes.c_int),
                ("d", ctypes.c_int), ("d_down", ctypes.c_int), ("w", ctypes.c_int),
                ("dtype", ctypes.c_int)]


class DarCacheStruct(ctypes.Structure):
    _fields_ = [("k_win", ctypes.c_void_p), ("v_win", ctypes.c_void_p),
                ("k_lat", ctypes.c_void_p), ("v_lat", ctypes.c_void_p),
                ("cap", ctypes.c_int), ("len", ctypes.c_int)]


class DarRopeStruct(ctypes.Structure):
    _fields_ = [("rotary_dim", ctypes.c_int), ("n_pos", ctypes.c_int),
                ("table", ctypes.c_void_p)]


class DarPagedCacheStruct(ctypes.Structure):
    _fields_ = [("k_win", ctypes.c_void_p), ("v_win", ctypes.c_void_p),
                ("k_pool", ctypes.c_void_p), ("v_pool", ctypes.c_void_p),
                ("block_table", ctypes.c_void_p), ("lens", ctypes.c_void_p),
                ("page_size", ctypes.c_int), ("max_blocks", ctypes.c_int), ("n_pages", ctypes.c_int)]


class DarError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__("%s: %s (status %d)" % (where, status_string(status), status))


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError("libdar.so is not built; run `python paper_2606_18587_amd/build.py` "
                          "(there is no non-HIP fallback)")
    lib = ctypes.CDLL(LIB_PATH)
    vp, sz, ci = ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int
    shp = ctypes.POINTER(DarShape)
    cp = ctypes.POINTER(DarCacheStruct)
    lib.dar_attn_prefill.restype = ci
    lib.dar_attn_prefill.argtypes = [shp, ci, vp, vp, vp, vp, vp, vp, vp, sz, vp]
    lib.dar_attn_prefill_lse.restype = ci
    lib.dar_attn_prefill_lse.argtypes = [shp, ci, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
    lib.dar_cache_append.restype = ci
    lib.dar_cache_append.argtypes = [shp, cp, vp, vp, ci, vp, vp]
    lib.dar_attn_decode.restype = ci
    lib.dar_attn_decode.argtypes = [shp, cp, vp, vp, vp, vp, vp, sz, vp]
    lib.dar_prefill_workspace_bytes.restype = sz
    lib.dar_prefill_workspace_bytes.argtypes = [shp, ci]
    lib.dar_decode_workspace_bytes.restype = sz
    lib.dar_decode_workspace_bytes.argtypes = [shp, ci]
    lib.dar_attn_prefill_backward.restype = ci
    lib.dar_attn_prefill_backward.argtypes = [shp, ci] + [vp] * 14 + [sz, vp]
    lib.dar_prefill_backward_workspace_bytes.restype = sz
    lib.dar_prefill_backward_workspace_bytes.argtypes = [shp, ci]
    lib.dar_attn_prefill_chunk.restype = ci
    lib.dar_attn_prefill_chunk.argtypes = [shp, cp, ci] + [vp] * 8 + [sz, vp]
    lib.dar_prefill_chunk_workspace_bytes.restype = sz
    lib.dar_prefill_chunk_workspace_bytes.argtypes = [shp, ci, ci]
    rp = ctypes.POINTER(DarRopeStruct)
    lib.dar_rope_table.restype = ci
    lib.dar_rope_table.argtypes = [ci, ctypes.c_double, ci, vp, vp]
    lib.dar_attn_prefill_rope.restype = ci
    lib.dar_attn_prefill_rope.argtypes = [shp, ci, ci, rp] + [vp] * 8 + [sz, vp]
    lib.dar_attn_prefill_rope_backward.restype = ci
    lib.dar_attn_prefill_rope_backward.argtypes = [shp, ci, ci, rp] + [vp] * 14 + [sz, vp]
    lib.dar_prefill_rope_backward_workspace_bytes.restype = sz
    lib.dar_prefill_rope_backward_workspace_bytes.argtypes = [shp, ci]
    lib.dar_attn_decode_rope.restype = ci
    lib.dar_attn_decode_rope.argtypes = [shp, cp, rp] + [vp] * 5 + [sz, vp]
    lib.dar_attn_prefill_shared.restype = ci
    lib.dar_attn_prefill_shared.argtypes = [shp, ci] + [vp] * 9 + [sz, vp]
    lib.dar_cache_append_shared.restype = ci
    lib.dar_cache_append_shared.argtypes = [shp, cp, vp, vp, vp, ci, vp]
    lib.dar_attn_decode_shared.restype = ci
    lib.dar_attn_decode_shared.argtypes = [shp, cp] + [vp] * 5 + [sz, vp]
    pcp = ctypes.POINTER(DarPagedCacheStruct)
    lib.dar_cache_append_paged.restype = ci
    lib.dar_cache_append_paged.argtypes = [shp, pcp, vp, vp, vp, vp]
    lib.dar_attn_decode_paged.restype = ci
    lib.dar_attn_decode_paged.argtypes = [shp, pcp] + [vp] * 5 + [sz, vp]
    lib.dar_attn_decode_paged_rope.restype = ci
    lib.dar_attn_decode_paged_rope.argtypes = [shp, pcp, rp] + [vp] * 5 + [sz, vp]
    lib.dar_attn_prefill_chunk_paged.restype = ci
    lib.dar_attn_prefill_chunk_paged.argtypes = [shp, pcp, ci] + [vp] * 9 + [sz, vp]
    lib.dar_prefill_chunk_paged_workspace_bytes.restype = sz
    lib.dar_prefill_chunk_paged_workspace_bytes.argtypes = [shp, ci, ci]
    lib.dar_attn_prefill_ragged.restype = ci
    lib.dar_attn_prefill_ragged.argtypes = [shp, ci] + [vp] * 9 + [sz, vp]
    lib.dar_prefill_rope_workspace_bytes.restype = sz
    lib.dar_prefill_rope_workspace_bytes.argtypes = [shp, ci]
    lib.dar_attn_prefill_chunk_rope.restype = ci
    lib.dar_attn_prefill_chunk_rope.argtypes = [shp, cp, rp, ci] + [vp] * 8 + [sz, vp]
    lib.dar_prefill_chunk_rope_workspace_bytes.restype = sz
    lib.dar_prefill_chunk_rope_workspace_bytes.argtypes = [shp, ci, ci]
    lib.dar_attn_decode_noalloc.restype = ci
    lib.dar_attn_decode_noalloc.argtypes = [shp, cp, vp, vp, vp, vp, vp]
    lib.dar_decode_noalloc_bytes.restype = sz
    lib.dar_decode_noalloc_bytes.argtypes = [shp, ci]
    lib.dar_decode_noalloc_max_bytes.restype = sz
    lib.dar_decode_noalloc_max_bytes.argtypes = []
    lib.dar_status_string.restype = ctypes.c_char_p
    lib.dar_status_string.argtypes = [ci]
    return lib


lib = _load()

EXPORTS = ("dar_attn_prefill", "dar_cache_append", "dar_attn_decode",
           "dar_attn_prefill_backward", "dar_prefill_workspace_bytes",
           "dar_decode_workspace_bytes", "dar_prefill_backward_workspace_bytes",
           "dar_status_string")


def status_string(st: int) -> str:
    return lib.dar_status_string(int(st)).decode()


def _dtype_code(t: torch.dtype) -> int:
    if t == torch.float32:
        return DAR_F32
    if t == torch.bfloat16:
        return DAR_BF16
    raise TypeError("DAR tensors must be float32 or bfloat16, got %s" % t)


def _ptr(t):
    if t is None:
        return None
    if not t.is_contiguous():
        raise ValueError("DAR tensors must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def make_shape(B, Hq, Hkv, d, d_down, w, dtype) -> DarShape:
    return DarShape(int(B), int(Hq), int(Hkv), int(d), int(d_down), int(w), _dtype_code(dtype))


def dar_prefill_workspace_bytes(shape: DarShape, T: int) -> int:
    return int(lib.dar_prefill_workspace_bytes(ctypes.byref(shape), int(T)))


def dar_decode_workspace_bytes(shape: DarShape, cap: int) -> int:
    return int(lib.dar_decode_workspace_bytes(ctypes.byref(shape), int(cap)))


def dar_prefill_backward_workspace_bytes(shape: DarShape, T: int) -> int:
    return int(lib.dar_prefill_backward_workspace_bytes(ctypes.byref(shape), int(T)))


def dar_status_string(st: int) -> str:
    return status_string(st)


def _workspace(nbytes, device):
    if nbytes == 0:
        return None
    return torch.empty(nbytes, dtype=torch.uint8, device=device)


def dar_attn_prefill(q, k, v, w_down, w_up, w, o=None, ws=None, stream=None, check=True,
                     lse=None, return_lse=False):
    """Causal DAR prefill. q [B,Hq,T,d]; k, v [B,Hkv,T,d]; w_down [Hkv,d,dd];
    w_up [Hkv,dd,d] or None (tied). Returns o [B,Hq,T,d], or (o, lse) with
    return_lse (lse [B,Hq,T] fp32, the log of each row's softmax denominator,
    written into `lse` when given). Calls dar_attn_prefill, or
    dar_attn_prefill_lse when the log-sum-exp is asked for."""
    B, Hq, T, d = q.shape
    Hkv = k.shape[1]
    dd = w_down.shape[2]
    shape = make_shape(B, Hq, Hkv, d, dd, w, q.dtype)
    if check:
        for name, t, want in (("k", k, (B, Hkv, T, d)), ("v", v, (B, Hkv, T, d)),
                              ("w_down", w_down, (Hkv, d, dd))):
            if tuple(t.shape) != want or t.dtype != q.dtype:
                raise ValueError("%s: expected %s %s, got %s %s" % (name, want, q.dtype,
                                                                   tuple(t.shape), t.dtype))
        if w_up is not None and (tuple(w_up.shape) != (Hkv, dd, d) or w_up.dtype != q.dtype):
            raise ValueError("w_up: expected %s" % ((Hkv, dd, d),))
    if o is None:
        o = torch.empty_like(q)
    if return_lse and lse is None:
        lse = torch.empty(B, Hq, T, dtype=torch.float32, device=q.device)
    if lse is not None and (tuple(lse.shape) != (B, Hq, T) or lse.dtype != torch.float32):
        raise ValueError("lse: expected %s float32" % ((B, Hq, T),))
    need = dar_prefill_workspace_bytes(shape, T)
    if ws is None:
        ws = _workspace(need, q.device)
    wsb = 0 if ws is None else ws.numel() * ws.element_size()
    if lse is None:
        st = lib.dar_attn_prefill(ctypes.byref(shape), int(T), _ptr(q), _ptr(k), _ptr(v),
                                  _ptr(w_down), _ptr(w_up), _ptr(o), _ptr(ws), wsb,
                                  _stream(stream))
        where = "dar_attn_prefill"
    else:
        st = lib.dar_attn_prefill_lse(ctypes.byref(shape), int(T), _ptr(q), _ptr(k), _ptr(v),
                                      _ptr(w_down), _ptr(w_up), _ptr(o), _ptr(lse), _ptr(ws),
                                      wsb, _stream(stream))
        where = "dar_attn_prefill_lse"
    if st != DAR_OK:
        raise DarError(st, where)
    return (o, lse) if return_lse else o


def dar_attn_prefill_lse(q, k, v, w_down, w_up, w, o=None, lse=None, ws=None, stream=None,
                         check=True):
    """dar_attn_prefill that also returns each row's log-sum-exp: (o, lse),
    lse [B,Hq,T] fp32 (written into `lse` when given)."""
    return dar_attn_prefill(q, k, v, w_down, w_up, w, o=o, ws=ws, stream=stream, check=check,
                            lse=lse, return_lse=True)


def dar_rope_table(rotary_dim, base, n_pos, device="cuda", stream=None):
    """The angle table [n_pos, rotary_dim] fp32: cos of the r/2 angles of each
    position, then their sin (computed on the device in fp64)."""
    table = torch.empty(int(n_pos), int(rotary_dim), dtype=torch.float32, device=device)
    st = lib.dar_rope_table(int(rotary_dim), float(base), int(n_pos), _ptr(table), _stream(stream))
    if st != DAR_OK:
        raise DarError(st, "dar_rope_table")
    return table


class Rope:
    """Rotary embedding of Eq. 3: rotate-half pairs over the first rotary_dim
    elements, angle p * base^(-2m/r); `table` [n_pos, r] fp32 on the device
    (filled by dar_rope_table unless given)."""

    def __init__(self, rotary_dim, base=10000.0, n_pos=4096, device="cuda", table=None,
                 stream=None):
        self.rotary_dim = int(rotary_dim)
        self.base = float(base)
        self.n_pos = int(n_pos)
        if table is None and self.rotary_dim > 0:
            table = dar_rope_table(self.rotary_dim, self.base, self.n_pos, device, stream)
        self.table = table

    def struct(self) -> DarRopeStruct:
        return DarRopeStruct(self.rotary_dim, self.n_pos,
                             None if self.table is None else self.table.data_ptr())


def dar_prefill_rope_workspace_bytes(shape: DarShape, T: int) -> int:
    return int(lib.dar_prefill_rope_workspace_bytes(ctypes.byref(shape), int(T)))


def dar_attn_prefill_rope(q, k, v, w_down, w_up, w, rope: Rope, pos0=0, o=None, ws=None,
                          stream=None, check=True, lse=None, return_lse=False):
    """Causal DAR prefill with the rotary embedding of Eq. 3 at positions
    pos0..pos0+T-1; q, k un-rotated. Other arguments as dar_attn_prefill."""
    B, Hq, T, d = q.shape
    Hkv = k.shape[1]
    dd = w_down.shape[2]
    shape = make_shape(B, Hq, Hkv, d, dd, w, q.dtype)
    if check:
        for name, t, want in (("k", k, (B, Hkv, T, d)), ("v", v, (B, Hkv, T, d)),
                              ("w_down", w_down, (Hkv, d, dd))):
            if tuple(t.shape) != want or t.dtype != q.dtype:
                raise ValueError("%s: expected %s %s, got %s %s" % (name, want, q.dtype,
                                                                   tuple(t.shape), t.dtype))
        if w_up is not None and (tuple(w_up.shape) != (Hkv, dd, d) or w_up.dtype != q.dtype):
            raise ValueError("w_up: expected %s" % ((Hkv, dd, d),))
    if o is None:
        o = torch.empty_like(q)
    if return_lse and lse is None:
        lse = torch.empty(B, Hq, T, dtype=torch.float32, device=q.device)
    if lse is not None and (tuple(lse.shape) != (B, Hq, T) or lse.dtype != torch.float32):
        raise ValueError("lse: expected %s float32" % ((B, Hq, T),))
    if ws is None:
        ws = _workspace(dar_prefill_rope_workspace_bytes(shape, T), q.device)
    rs = rope.struct()
    st = lib.dar_attn_prefill_rope(ctypes.byref(shape), int(T), int(pos0), ctypes.byref(rs),
                                   _ptr(q), _ptr(k), _ptr(v), _ptr(w_down), _ptr(w_up), _ptr(o),
                                   _ptr(lse), _ptr(ws),
                                   0 if ws is None else ws.numel() * ws.element_size(),
                                   _stream(stream))
    if st != DAR_OK:
        raise DarError(st, "dar_attn_prefill_rope")
    return (o, lse) if return_lse else o


def dar_attn_prefill_backward(q, k, v, w_down, w_up, w, o, lse, dout, ws=None, stream=None,
                              check=True):
    """Gradients of sum(dout * o) of the causal DAR prefill, given the forward's
    o and lse (dar_attn_prefill(..., return_lse=True)). Returns
    (dq, dk, dv, dw_down, dw_up): dq/dk/dv in the input dtype, the weight
    gradients fp32; dw_up is None when tied (w_up None), dw_down then holds the
    gradient of the shared matrix."""
    B, Hq, T, d = q.shape
    Hkv = k.shape[1]
    dd = w_down.shape[2]
    shape = make_shape(B, Hq, Hkv, d, dd, w, q.dtype)
    if check:
        for name, t, want in (("k", k, (B, Hkv, T, d)), ("v", v, (B, Hkv, T, d)),
                              ("w_down", w_down, (Hkv, d, dd)), ("o", o, (B, Hq, T, d)),
                              ("dout", dout, (B, Hq, T, d))):
            if tuple(t.shape) != want or t.dtype != q.dtype:
                raise ValueError("%s: expected %s %s, got %s %s" % (name, want, q.dtype,
                                                                   tuple(t.shape), t.dtype))
        if w_up is not None and (tuple(w_up.shape) != (Hkv, dd, d) or w_up.dtype != q.dtype):
            raise ValueError("w_up: expected %s" % ((Hkv, dd, d),))
        if tuple(lse.shape) != (B, Hq, T) or lse.dtype != torch.float32:
            raise ValueError("lse: expected %s float32" % ((B, Hq, T),))
    dq = torch.empty_like(q)
    dk = torch.empty_like(k)
    dv = torch.empty_like(v)
    dwd = torch.empty(Hkv, d, dd, dtype=torch.float32, device=q.device)
    dwu = None if w_up is None else torch.empty(Hkv, dd, d, dtype=torch.float32, device=q.device)
    if ws is None:
        ws = _workspace(dar_prefill_backward_workspace_bytes(shape, T), q.device)
    st = lib.dar_attn_prefill_backward(ctypes.byref(shape), int(T), _ptr(q), _ptr(k), _ptr(v),
                                       _ptr(w_down), _ptr(w_up), _ptr(o), _ptr(lse), _ptr(dout),
                                       _ptr(dq),
                                       _ptr(dk), _ptr(dv), _ptr(dwd), _ptr(dwu), _ptr(ws),
                                       0 if ws is None else ws.numel() * ws.element_size(),
                                       _stream(stream))
    if st != DAR_OK:
        raise DarError(st, "dar_attn_prefill_backward")
    return dq, dk, dv, dwd, dwu


def dar_prefill_rope_backward_workspace_bytes(shape: DarShape, T: int) -> int:
    return int(lib.dar_prefill_rope_backward_workspace_bytes(ctypes.byref(shape), int(T)))


def dar_attn_prefill_rope_backward(q, k, v, w_down, w_up, w, rope: "Rope", o, lse, dout, pos0=0,
                                   ws=None, stream=None):
    """Gradients of sum(dout * o) of dar_attn_prefill_rope (same q, k, v,
    weights, rope and pos0; its o and lse). Returns (dq, dk, dv, dw_down,
    dw_up) as dar_attn_prefill_backward does."""
    B, Hq, T, d = q.shape
    Hkv = k.shape[1]
    dd = w_down.shape[2]
    shape = make_shape(B, Hq, Hkv, d, dd, w, q.dtype)
    for name, t, want in (("k", k, (B, Hkv, T, d)), ("v", v, (B, Hkv, T, d)),
                          ("w_down", w_down, (Hkv, d, dd)), ("o", o, (B, Hq, T, d)),
                          ("dout", dout, (B, Hq, T, d))):
        if tuple(t.shape) != want or t.dtype != q.dtype:
            raise ValueError("%s: expected %s %s" % (name, want, q.dtype))
    if tuple(lse.shape) != (B, Hq, T) or lse.dtype != torch.float32:
        raise ValueError("lse: expected %s float32" % ((B, Hq, T),))
    dq = torch.empty_like(q)
    dk = torch.empty_like(k)
    dv = torch.empty_like(v)
    dwd = torch.empty(Hkv, d, dd, dtype=torch.float32, device=q.device)
    dwu = None if w_up is None else torch.empty(Hkv, dd, d, dtype=torch.float32, device=q.device)
    if ws is None:
        ws = _workspace(dar_prefill_rope_backward_workspace_bytes(shape, T), q.device)
    rs = rope.struct()
    st = lib.dar_attn_prefill_rope_backward(ctypes.byref(shape), int(T), int(pos0), ctypes.byref(rs),
                                            _ptr(q), _ptr(k), _ptr(v), _ptr(w_down), _ptr(w_up),
                                            _ptr(o), _ptr(lse), _ptr(dout), _ptr(dq), _ptr(dk),
                                            _ptr(dv), _ptr(dwd), _ptr(dwu), _ptr(ws),
                                            0 if ws is None else ws.numel() * ws.element_size(),
                                            _stream(stream))
    if st != DAR_OK:
        raise DarError(st, "dar_attn_prefill_rope_backward")
    return dq, dk, dv, dwd, dwu


class DarCache:
    """Split KV cache owned by torch: ring [B,Hkv,w,d] for the window and
    latents [B,Hkv,cap,dd] for older tokens (see dar_cache in include/dar.h)."""

    def __init__(self, B, Hkv, d, d_down, w, cap, dtype, device="cuda", shared=False):
        """shared: one latent array (the single shared latent per token; used
        with the *_shared entry points), else separate key and value latents."""
        self.B, self.Hkv, self.d, self.d_down, self.w, self.cap = B, Hkv, d, d_down, w, cap
        self.dtype = dtype
        self.shared = shared
        wl = max(w, 1)  # keep valid pointers for w = 0 (the ring is never touched then)
        self.k_win = torch.zeros(B, Hkv, wl, d, dtype=dtype, device=device)
        self.v_win = torch.zeros(B, Hkv, wl, d, dtype=dtype, device=device)
        self.k_lat = torch.zeros(B, Hkv, cap, d_down, dtype=dtype, device=device)
        self.v_lat = self.k_lat if shared else torch.zeros(B, Hkv, cap, d_down, dtype=dtype,
                                                           device=device)
        self.struct = DarCacheStruct(self.k_win.data_ptr(), self.v_win.data_ptr(),
                                     self.k_lat.data_ptr(), self.v_lat.data_ptr(), int(cap), 0)

    @property
    def len(self) -> int:
        return int(self.struct.len)


def dar_cache_append(cache: DarCache, k_new, v_new, w_down, Hq=None, stream=None):
    """Append n tokens k_new, v_new [B,Hkv,n,d]; projects window exits to latents."""
    B, Hkv, n, d = k_new.shape
    shape = make_shape(B, Hq if Hq is not None else Hkv, Hkv, d, cache.d_down, cache.w,
                       k_new.dtype)
    if tuple(v_new.shape) != (B, Hkv, n, d) or (B, Hkv, d) != (cache.B, cache.Hkv, cache.d):
        raise ValueError("k_new/v_new do not match the cache")
    st = lib.dar_cache_append(ctypes.byref(shape), ctypes.byref(cache.struct), _ptr(k_new),
                              _ptr(v_new), int(n), _ptr(w_down), _stream(stream))
    if st != DAR_OK:
        raise DarError(st, "dar_cache_append")
    return cache


def dar_prefill_chunk_workspace_bytes(shape, len_, n) -> int:
    return int(lib.dar_prefill_chunk_workspace_bytes(ctypes.byref(shape), int(len_), int(n)))


def dar_attn_prefill_chunk(cache: DarCache, q, k_new, v_new, w_down, w_up=None, o=None,
                           lse=None, return_lse=False, ws=None, stream=None, check=True):
    """Chunked prefill: n new tokens (q [B,Hq,n,d], k_new/v_new [B,Hkv,n,d]) at
    positions cache.len.. attend to everything before them (ring + latents of the
    cache, and each other, causally); then the cache is extended by them as
    dar_cache_append would. Returns o [B,Hq,n,d], or (o, lse) with return_lse."""
    B, Hq, n, d = q.shape
    Hkv = cache.Hkv
    shape = make_shape(B, Hq, Hkv, d, cache.d_down, cache.w, q.dtype)
    if check:
        for name, t in (("k_new", k_new), ("v_new", v_new)):
            if tuple(t.shape) != (B, Hkv, n, d) or t.dtype != q.dtype:
                raise ValueError("%s: expected %s %s" % (name, (B, Hkv, n, d), q.dtype))
        if (B, d) != (cache.B, cache.d) or q.dtype != cache.dtype:
            raise ValueError("q does not match the cache")
    if o is None:
        o = torch.empty_like(q)
    if return_lse and lse is None:
        lse = torch.empty(B, Hq, n, dtype=torch.float32, device=q.device)
    if ws is None:
        ws = _workspace(dar_prefill_chunk_workspace_bytes(shape, cache.len, n), q.device)
    st = lib.dar_attn_prefill_chunk(ctypes.byref(shape), ctypes.byref(cache.struct), int(n),
                                    _ptr(q), _ptr(k_new), _ptr(v_new), _ptr(w_down), _ptr(w_up),
                                    _ptr(o), _ptr(lse), _ptr(ws),
                                    0 if ws is None else ws.numel() * ws.element_size(),
                                    _stream(stream))
    if st != DAR_OK:
        raise DarError(st, "dar_attn_prefill_chunk")
    return (o, lse) if return_lse else o


def dar_prefill_chunk_rope_workspace_bytes(shape, len_, n) -> int:
    return int(lib.dar_prefill_chunk_rope_workspace_bytes(ctypes.byref(shape), int(len_), int(n)))


def dar_attn_prefill_chunk_rope(cache: DarCache, q, k_new, v_new, w_down, rope: "Rope", w_up=None,
                                o=None, lse=None, return_lse=False, ws=None, stream=None,
                                check=True):
    """Chunked prefill with the rotary embedding of Eq. 3: n new tokens at
    positions cache.len.. (q, k_new, v_new un-rotated, shapes as
    dar_attn_prefill_chunk); the cache is extended by the un-rotated tokens.
    Returns o [B,Hq,n,d], or (o, lse) with return_lse."""
    B, Hq, n, d = q.shape
    Hkv = cache.Hkv
    shape = make_shape(B, Hq, Hkv, d, cache.d_down, cache.w, q.dtype)
    if check:
        for name, t in (("k_new", k_new), ("v_new", v_new)):
            if tuple(t.shape) != (B, Hkv, n, d) or t.dtype != q.dtype:
                raise ValueError("%s: expected %s %s" % (name, (B, Hkv, n, d), q.dtype))
        if (B, d) != (cache.B, cache.d) or q.dtype != cache.dtype:
            raise ValueError("q does not match the cache")
    if o is None:
        o = torch.empty_like(q)
    if return_lse and lse is None:
        lse = torch.empty(B, Hq, n, dtype=torch.float32, device=q.device)
    if ws is None:
        ws = _workspace(dar_prefill_chunk_rope_workspace_bytes(shape, cache.len, n), q.device)
    rs = rope.struct()
    st = lib.dar_attn_prefill_chunk_rope(ctypes.byref(shape), ctypes.byref(cache.struct),
                                         ctypes.byref(rs), int(n), _ptr(q), _ptr(k_new),
                                         _ptr(v_new), _ptr(w_down), _ptr(w_up), _ptr(o),
                                         _ptr(lse), _ptr(ws),
                                         0 if ws is None else ws.numel() * ws.element_size(),
                                         _stream(stream))
    if st != DAR_OK:
        raise DarError(st, "dar_attn_prefill_chunk_rope")
    return (o, lse) if return_lse else o


def dar_attn_decode(cache: DarCache, q, w_down, w_up=None, o=None, ws=None, stream=None):
    """One decode step: q [B,Hq,d] at position cache.len - 1. Returns o [B,Hq,d]."""
    B, Hq, d = q.shape
    shape = make_shape(B, Hq, cache.Hkv, d, cache.d_down, cache.w, q.dtype)
    if o is None:
        o = torch.empty_like(q)
    if ws is None:
        ws = _workspace(dar_decode_workspace_bytes(shape, cache.cap), q.device)
    st = lib.dar_attn_decode(ctypes.byref(shape), ctypes.byref(cache.struct), _ptr(q),
                             _ptr(w_down), _ptr(w_up), _ptr(o), _ptr(ws),
                             0 if ws is None else ws.numel() * ws.element_size(),
                             _stream(stream))
    if st != DAR_OK:
        raise DarError(st, "dar_attn_decode")
    return o


def dar_attn_decode_noalloc(cache: "DarCache", q, w_down, w_up=None, o=None, stream=None):
    """One decode step as dar_attn_decode, through the entry point that takes
    no workspace (its partial records live in a fixed array inside the
    library). Pass `o` to keep the call free of allocation."""
    B, Hq, d = q.shape
    shape = make_shape(B, Hq, cache.Hkv, d, cache.d_down, cache.w, q.dtype)
    if o is None:
        o = torch.empty_like(q)
    st = lib.dar_attn_decode_noalloc(ctypes.byref(shape), ctypes.byref(cache.struct), _ptr(q),
                                     _ptr(w_down), _ptr(w_up), _ptr(o), _stream(stream))
    if st != DAR_OK:
        raise DarError(st, "dar_attn_decode_noalloc")
    return o


def dar_decode_noalloc_bytes(shape: DarShape, length: int) -> int:
    return int(lib.dar_decode_noalloc_bytes(ctypes.byref(shape), int(length)))


def dar_decode_noalloc_max_bytes() -> int:
    return int(lib.dar_decode_noalloc_max_bytes())


def dar_attn_decode_rope(cache: "DarCache", q, w_down, rope: Rope, w_up=None, o=None, ws=None,
                         stream=None):
    """One decode step with the rotary embedding of Eq. 3; q [B,Hq,d] un-rotated,
    at position cache.len - 1. Returns o [B,Hq,d]."""
    B, Hq, d = q.shape
    shape = make_shape(B, Hq, cache.Hkv, d, cache.d_down, cache.w, q.dtype)
    if o is None:
        o = torch.empty_like(q)
    if ws is None:
        ws = _workspace(dar_decode_workspace_bytes(shape, cache.cap), q.device)
    rs = rope.struct()
    st = lib.dar_attn_decode_rope(ctypes.byref(shape), ctypes.byref(cache.struct), ctypes.byref(rs), _ptr(q),
                                  _ptr(w_down), _ptr(w_up), _ptr(o), _ptr(ws),
                                  0 if ws is None else ws.numel() * ws.element_size(),
                                  _stream(stream))
    if st != DAR_OK:
        raise DarError(st, "dar_attn_decode_rope")
    return o


def dar_attn_prefill_shared(q, k, v, c, u_k, u_v, w, o=None, ws=None, stream=None, lse=None,
                            return_lse=False):
    """Causal prefill with one shared latent per token: c [B,Hkv,T,dd]; distant
    key c U_K, distant value c U_V (u_k, u_v [Hkv,dd,d])."""
    B, Hq, T, d = q.shape
    Hkv = k.shape[1]
    dd = c.shape[3]
    shape = make_shape(B, Hq, Hkv, d, dd, w, q.dtype)
    for name, t, want in (("k", k, (B, Hkv, T, d)), ("v", v, (B, Hkv, T, d)),
                          ("c", c, (B, Hkv, T, dd)), ("u_k", u_k, (Hkv, dd, d)),
                          ("u_v", u_v, (Hkv, dd, d))):
        if tuple(t.shape) != want or t.dtype != q.dtype:
            raise ValueError("%s: expected %s %s" % (name, want, q.dtype))
    if o is None:
        o = torch.empty_like(q)
    if return_lse and lse is None:
        lse = torch.empty(B, Hq, T, dtype=torch.float32, device=q.device)
    if ws is None:
        ws = _workspace(dar_prefill_workspace_bytes(shape, T), q.device)
    st = lib.dar_attn_prefill_shared(ctypes.byref(shape), int(T), _ptr(q), _ptr(k), _ptr(v), _ptr(c),
                                     _ptr(u_k), _ptr(u_v), _ptr(o), _ptr(lse), _ptr(ws),
                                     0 if ws is None else ws.numel() * ws.element_size(),
                                     _stream(stream))
    if st != DAR_OK:
        raise DarError(st, "dar_attn_prefill_shared")
    return (o, lse) if return_lse else o


def dar_cache_append_shared(cache: DarCache, k_new, v_new, c_new, Hq=None, stream=None):
    """Append n tokens with their shared latents c_new [B,Hkv,n,dd]."""
    assert cache.shared, "a cache made with shared=True"
    B, Hkv, n, d = k_new.shape
    shape = make_shape(B, Hq or Hkv, Hkv, d, cache.d_down, cache.w, k_new.dtype)
    st = lib.dar_cache_append_shared(ctypes.byref(shape), ctypes.byref(cache.struct), _ptr(k_new),
                                     _ptr(v_new), _ptr(c_new), int(n), _stream(stream))
    if st != DAR_OK:
        raise DarError(st, "dar_cache_append_shared")


def dar_attn_decode_shared(cache: DarCache, q, u_k, u_v, o=None, ws=None, stream=None):
    """One decode step over a shared-latent cache; q [B,Hq,d] at position len-1."""
    assert cache.shared, "a cache made with shared=True"
    B, Hq, d = q.shape
    shape = make_shape(B, Hq, cache.Hkv, d, cache.d_down, cache.w, q.dtype)
    if o is None:
        o = torch.empty_like(q)
    if ws is None:
        ws = _workspace(dar_decode_workspace_bytes(shape, cache.cap), q.device)
    st = lib.dar_attn_decode_shared(ctypes.byref(shape), ctypes.byref(cache.struct), _ptr(q),
                                    _ptr(u_k), _ptr(u_v), _ptr(o), _ptr(ws),
                                    0 if ws is None else ws.numel() * ws.element_size(),
                                    _stream(stream))
    if st != DAR_OK:
        raise DarError(st, "dar_attn_decode_shared")
    return o


class DarPagedCache:
    """Paged split cache (include/dar.h, dar_paged_cache): rings [B,Hkv,w,d],
    latent pages [n_pages,Hkv,page_size,dd] for keys and values, a block table
    [B,max_blocks] (int32, device) and per-sequence lengths [B] (int32,
    device). block_table and lens are plain torch tensors the caller fills."""

    def __init__(self, B, Hkv, d, d_down, w, page_size, max_blocks, n_pages, dtype,
                 device="cuda"):
        self.B, self.Hkv, self.d, self.d_down, self.w = B, Hkv, d, d_down, w
        self.page_size, self.max_blocks, self.n_pages = page_size, max_blocks, n_pages
        wl = max(w, 1)
        self.k_win = torch.zeros(B, Hkv, wl, d, dtype=dtype, device=device)
        self.v_win = torch.zeros(B, Hkv, wl, d, dtype=dtype, device=device)
        self.k_pool = torch.zeros(n_pages, Hkv, page_size, d_down, dtype=dtype, device=device)
        self.v_pool = torch.zeros(n_pages, Hkv, page_size, d_down, dtype=dtype, device=device)
        self.block_table = torch.full((B, max_blocks), -1, dtype=torch.int32, device=device)
        self.lens = torch.zeros(B, dtype=torch.int32, device=device)

    @property
    def cap(self):
        return self.page_size * self.max_blocks

    def overflowed(self):
        """Sequences the append found at capacity (lens marked -1 - n); reads
        lens back to the host (synchronises with the current stream)."""
        return [b for b, n in enumerate(self.lens.cpu().tolist()) if n < 0]

    def struct(self) -> DarPagedCacheStruct:
        return DarPagedCacheStruct(self.k_win.data_ptr(), self.v_win.data_ptr(),
                                   self.k_pool.data_ptr(), self.v_pool.data_ptr(),
                                   self.block_table.data_ptr(), self.lens.data_ptr(),
                                   self.page_size, self.max_blocks, self.n_pages)


def dar_cache_append_paged(cache: DarPagedCache, k_new, v_new, w_down, Hq=None, stream=None):
    """One token per sequence: k_new, v_new [B,Hkv,d]; lens advance on the device."""
    B, Hkv, d = k_new.shape
    shape = make_shape(B, Hq or Hkv, Hkv, d, cache.d_down, cache.w, k_new.dtype)
    cs = cache.struct()
    st = lib.dar_cache_append_paged(ctypes.byref(shape), ctypes.byref(cs), _ptr(k_new), _ptr(v_new),
                                    _ptr(w_down), _stream(stream))
    if st != DAR_OK:
        raise DarError(st, "dar_cache_append_paged")


def dar_attn_decode_paged(cache: DarPagedCache, q, w_down, w_up=None, o=None, ws=None, stream=None):
    """One decode step per sequence (query at position lens[b] - 1)."""
    B, Hq, d = q.shape
    shape = make_shape(B, Hq, cache.Hkv, d, cache.d_down, cache.w, q.dtype)
    if o is None:
        o = torch.empty_like(q)
    if ws is None:
        ws = _workspace(dar_decode_workspace_bytes(shape, cache.cap), q.device)
    cs = cache.struct()
    st = lib.dar_attn_decode_paged(ctypes.byref(shape), ctypes.byref(cs), _ptr(q), _ptr(w_down),
                                   _ptr(w_up), _ptr(o), _ptr(ws),
                                   0 if ws is None else ws.numel() * ws.element_size(),
                                   _stream(stream))
    if st != DAR_OK:
        raise DarError(st, "dar_attn_decode_paged")
    return o


def dar_attn_decode_paged_rope(cache: DarPagedCache, q, w_down, rope: "Rope", w_up=None, o=None,
                               ws=None, stream=None):
    """dar_attn_decode_paged with the rotary embedding of Eq. 3 (query of
    sequence b at position lens[b] - 1; rope.n_pos >= the cache capacity)."""
    B, Hq, d = q.shape
    shape = make_shape(B, Hq, cache.Hkv, d, cache.d_down, cache.w, q.dtype)
    if o is None:
        o = torch.empty_like(q)
    if ws is None:
        ws = _workspace(dar_decode_workspace_bytes(shape, cache.cap), q.device)
    cs = cache.struct()
    rs = rope.struct()
    st = lib.dar_attn_decode_paged_rope(ctypes.byref(shape), ctypes.byref(cs), ctypes.byref(rs),
                                        _ptr(q), _ptr(w_down), _ptr(w_up), _ptr(o), _ptr(ws),
                                        0 if ws is None else ws.numel() * ws.element_size(),
                                        _stream(stream))
    if st != DAR_OK:
        raise DarError(st, "dar_attn_decode_paged_rope")
    return o


def dar_prefill_chunk_paged_workspace_bytes(shape, cap, n) -> int:
    return int(lib.dar_prefill_chunk_paged_workspace_bytes(ctypes.byref(shape), int(cap), int(n)))


def dar_attn_prefill_chunk_paged(cache: DarPagedCache, q, k_new, v_new, w_down, w_up=None,
                                 n_new=None, o=None, lse=None, return_lse=False, ws=None,
                                 stream=None):
    """Chunked prefill over a paged cache: sequence b takes n_new[b] (device
    int32 [B], each <= n; None: all n) new tokens at positions lens[b]..,
    q [B,Hq,n,d], k_new/v_new [B,Hkv,n,d]; lens advance on the device.
    Returns o [B,Hq,n,d] (rows past n_new[b] not written), or (o, lse)."""
    B, Hq, n, d = q.shape
    Hkv = cache.Hkv
    shape = make_shape(B, Hq, Hkv, d, cache.d_down, cache.w, q.dtype)
    for name, t in (("k_new", k_new), ("v_new", v_new)):
        if tuple(t.shape) != (B, Hkv, n, d) or t.dtype != q.dtype:
            raise ValueError("%s: expected %s %s" % (name, (B, Hkv, n, d), q.dtype))
    if (B, d) != (cache.B, cache.d):
        raise ValueError("q does not match the cache")
    if n_new is not None and (n_new.dtype != torch.int32 or tuple(n_new.shape) != (B,)):
        raise ValueError("n_new: expected int32 [%d]" % B)
    if o is None:
        o = torch.empty_like(q)
    if return_lse and lse is None:
        lse = torch.empty(B, Hq, n, dtype=torch.float32, device=q.device)
    if ws is None:
        ws = _workspace(dar_prefill_chunk_paged_workspace_bytes(shape, cache.cap, n), q.device)
    cs = cache.struct()
    st = lib.dar_attn_prefill_chunk_paged(ctypes.byref(shape), ctypes.byref(cs), int(n),
                                          _ptr(n_new), _ptr(q), _ptr(k_new), _ptr(v_new),
                                          _ptr(w_down), _ptr(w_up), _ptr(o), _ptr(lse), _ptr(ws),
                                          0 if ws is None else ws.numel() * ws.element_size(),
                                          _stream(stream))
    if st != DAR_OK:
        raise DarError(st, "dar_attn_prefill_chunk_paged")
    return (o, lse) if return_lse else o


def dar_attn_prefill_ragged(q, k, v, w_down, w_up, w, seq_lens, o=None, ws=None, stream=None,
                            lse=None, return_lse=False):
    """Causal prefill of a padded batch whose sequence b holds seq_lens[b]
    tokens (int32 device tensor [B]); rows past a sequence's length are left
    unwritten. Other arguments as dar_attn_prefill."""
    B, Hq, T, d = q.shape
    Hkv = k.shape[1]
    dd = w_down.shape[2]
    shape = make_shape(B, Hq, Hkv, d, dd, w, q.dtype)
    if seq_lens.dtype != torch.int32 or tuple(seq_lens.shape) != (B,) or not seq_lens.is_cuda:
        raise ValueError("seq_lens: expected an int32 device tensor of shape (%d,)" % B)
    if o is None:
        o = torch.empty_like(q)
    if return_lse and lse is None:
        lse = torch.empty(B, Hq, T, dtype=torch.float32, device=q.device)
    if ws is None:
        ws = _workspace(dar_prefill_workspace_bytes(shape, T), q.device)
    st = lib.dar_attn_prefill_ragged(ctypes.byref(shape), int(T), _ptr(seq_lens), _ptr(q), _ptr(k),
                                     _ptr(v), _ptr(w_down), _ptr(w_up), _ptr(o), _ptr(lse), _ptr(ws),
                                     0 if ws is None else ws.numel() * ws.element_size(),
                                     _stream(stream))
    if st != DAR_OK:
        raise DarError(st, "dar_attn_prefill_ragged")
    return (o, lse) if return_lse else o
