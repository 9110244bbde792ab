"""The C ABI without a GPU: the library loads, exports every declared entry
point, sizes workspaces, and rejects bad arguments before touching HIP.

The rejection tests pass fake (never dereferenced) device addresses; they run
only where no GPU is visible, so a validation bug can never hand such an
address to a kernel.
"""
import ctypes
import os
import re

import pytest
import torch

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "dar.h")

dar = pytest.importorskip("paper_2606_18587_amd", reason="libdar.so not built")

no_gpu = pytest.mark.skipif(torch.cuda.is_available(),
                            reason="fake device addresses are only used where no GPU exists")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(dar_[a-z_]+)\s*\(", text)))


def test_exports_every_declared_symbol():
    names = declared_functions()
    assert set(names) == {"dar_attn_prefill", "dar_attn_prefill_lse", "dar_cache_append", "dar_attn_decode",
                          "dar_attn_prefill_backward", "dar_prefill_workspace_bytes",
                          "dar_decode_workspace_bytes", "dar_prefill_backward_workspace_bytes",
                          "dar_attn_prefill_chunk", "dar_prefill_chunk_workspace_bytes",
                          "dar_attn_prefill_chunk_rope", "dar_prefill_chunk_rope_workspace_bytes",
                          "dar_attn_prefill_chunk_paged", "dar_prefill_chunk_paged_workspace_bytes",
                          "dar_attn_prefill_rope_backward", "dar_prefill_rope_backward_workspace_bytes",
                          "dar_rope_table", "dar_attn_prefill_rope", "dar_attn_decode_rope",
                          "dar_attn_prefill_shared", "dar_cache_append_shared",
                          "dar_attn_decode_shared", "dar_cache_append_paged",
                          "dar_attn_decode_paged", "dar_attn_decode_paged_rope",
                          "dar_attn_prefill_ragged",
                          "dar_prefill_rope_workspace_bytes", "dar_status_string",
                          "dar_attn_decode_noalloc", "dar_decode_noalloc_bytes",
                          "dar_decode_noalloc_max_bytes"}
    raw = ctypes.CDLL(dar.LIB_PATH)
    for n in names:
        assert hasattr(raw, n), n


def test_k0_library_exports_its_header():
    """The microbenchmark library (include/dar_k0.h) loads without a GPU and
    exports what its header declares."""
    text = open(os.path.join(ROOT, "include", "dar_k0.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = sorted(set(re.findall(r"\b(dar_[a-z0-9_]+)\s*\(", text)))
    assert names == ["dar_k0_measure"]
    from paper_2606_18587_amd import k0
    raw = ctypes.CDLL(k0.K0_LIB_PATH)
    for n in names:
        assert hasattr(raw, n), n


@no_gpu
def test_k0_rejects_small_buffer():
    from paper_2606_18587_amd import k0
    lib = k0._load()
    r = k0.DarK0Result()
    assert lib.dar_k0_measure(FAKE, 1 << 20, ctypes.byref(r), None) == 1
    assert lib.dar_k0_measure(None, 1 << 31, ctypes.byref(r), None) == 1
    assert lib.dar_k0_measure(MISALIGNED, 1 << 31, ctypes.byref(r), None) == 1


def test_status_strings():
    for st in range(6):
        assert dar.status_string(st)
    assert dar.status_string(99) == "unknown status"


def S(B=2, Hq=4, Hkv=2, d=64, dd=16, w=8, dtype=torch.bfloat16):
    return dar.make_shape(B, Hq, Hkv, d, dd, w, dtype)


def expected_prefill_ws(B, Hkv, T, dd, w, esize):
    """Latent keys (Tp rows of dd) and transposed latent values (Tp/32 blocks
    of up to dd + 1 rows of 32) over Tp = round_up(T - w, 32) + 64 tokens (none
    when T <= w), per-32-token latent norms and key norms (fp32), 256 bytes of
    constant rows; every part 256-byte aligned."""
    al = lambda x: (x + 255) // 256 * 256
    Tp = (T - w + 31) // 32 * 32 + 64 if T > w else 0
    return (al(B * Hkv * Tp * dd * esize) + al(B * Hkv * Tp * (dd + 1) * esize)
            + al(B * Hkv * (Tp // 32) * 4) + al(B * Hkv * ((T + 31) // 32) * 4) + 256)


def test_prefill_workspace_size():
    s = S()
    assert dar.dar_prefill_workspace_bytes(s, 100) == expected_prefill_ws(2, 2, 100, 16, 8, 2)
    assert dar.dar_prefill_workspace_bytes(s, 8) == expected_prefill_ws(2, 2, 8, 16, 8, 2)
    assert dar.dar_prefill_workspace_bytes(s, 8) < 1024     # T <= w: no latents, only norms
    assert dar.dar_prefill_workspace_bytes(S(w=0, dtype=torch.float32), 64) == \
        expected_prefill_ws(2, 2, 64, 16, 0, 4)
    assert dar.dar_prefill_workspace_bytes(S(Hq=3), 64) == 0   # invalid shape


def test_decode_workspace_size_grows_with_capacity():
    s = S()
    a = dar.dar_decode_workspace_bytes(s, 1000)
    b = dar.dar_decode_workspace_bytes(s, 100000)
    assert 0 < a < b
    # whole partial records {m, l, acc_lat, acc_win} per (batch, query head),
    # then one int per (batch, KV head): the paged decode's record count
    rec = s.B * s.Hq * (2 + s.d_down + s.d) * 4
    for x in (a, b):
        assert (x - s.B * s.Hkv * 4) % rec == 0
    assert dar.dar_decode_workspace_bytes(S(Hq=12, Hkv=4), 100) == 0  # group of 3: unsupported


FAKE = ctypes.c_void_p(1 << 20)       # aligned, never dereferenced
MISALIGNED = ctypes.c_void_p((1 << 20) + 2)


def call_prefill(shape, T=16, q=FAKE, k=FAKE, v=FAKE, wd=FAKE, wu=None, o=FAKE, lse=None,
                 ws=FAKE, ws_bytes=1 << 30):
    if lse is None:
        st = dar.lib.dar_attn_prefill(ctypes.byref(shape), T, q, k, v, wd, wu, o, ws, ws_bytes,
                                      None)
        # the lse entry point with lse = NULL validates the same way
        assert dar.lib.dar_attn_prefill_lse(ctypes.byref(shape), T, q, k, v, wd, wu, o, None, ws,
                                            ws_bytes, None) == st
        return st
    return dar.lib.dar_attn_prefill_lse(ctypes.byref(shape), T, q, k, v, wd, wu, o, lse, ws,
                                        ws_bytes, None)


@no_gpu
@pytest.mark.parametrize("kw,shape_kw,expect", [
    ({}, {"Hq": 3}, dar.DAR_E_ARG),                 # Hq % Hkv != 0
    ({}, {"dd": 65}, dar.DAR_E_ARG),                # d_down > d
    ({}, {"w": -1}, dar.DAR_E_ARG),
    ({}, {"B": 0}, dar.DAR_E_ARG),
    ({}, {"d": 512, "dd": 16}, dar.DAR_E_UNSUPPORTED),
    ({"T": 0}, {}, dar.DAR_E_ARG),
    ({"q": None}, {}, dar.DAR_E_ARG),
    ({"k": MISALIGNED}, {}, dar.DAR_E_ARG),
    ({"wu": MISALIGNED}, {}, dar.DAR_E_ARG),
    ({"lse": MISALIGNED}, {}, dar.DAR_E_ARG),
    ({"ws": None, "ws_bytes": 0}, {}, dar.DAR_E_WORKSPACE),
    ({"ws_bytes": 16}, {}, dar.DAR_E_WORKSPACE),
])
def test_prefill_rejects(kw, shape_kw, expect):
    assert call_prefill(S(**shape_kw), **kw) == expect


@no_gpu
def test_prefill_bad_dtype():
    s = S()
    s.dtype = 7
    assert call_prefill(s) == dar.DAR_E_ARG


def cache_struct(cap=64, length=0, win=FAKE):
    return dar.DarCacheStruct(win.value if win else None, win.value if win else None,
                              FAKE.value, FAKE.value, cap, length)


@no_gpu
def test_append_capacity_and_arguments():
    s = S()
    c = cache_struct(cap=64, length=60)
    st = dar.lib.dar_cache_append(ctypes.byref(s), ctypes.byref(c), FAKE, FAKE, 5, FAKE, None)
    assert st == dar.DAR_E_CAPACITY and c.len == 60
    st = dar.lib.dar_cache_append(ctypes.byref(s), ctypes.byref(c), FAKE, FAKE, 0, FAKE, None)
    assert st == dar.DAR_E_ARG and c.len == 60
    st = dar.lib.dar_cache_append(ctypes.byref(s), ctypes.byref(c), MISALIGNED, FAKE, 1, FAKE,
                                  None)
    assert st == dar.DAR_E_ARG and c.len == 60
    c2 = cache_struct(win=None)  # a ring is required when w > 0
    st = dar.lib.dar_cache_append(ctypes.byref(s), ctypes.byref(c2), FAKE, FAKE, 1, FAKE, None)
    assert st == dar.DAR_E_ARG and c2.len == 0
    c3 = cache_struct(cap=64, length=65)
    st = dar.lib.dar_cache_append(ctypes.byref(s), ctypes.byref(c3), FAKE, FAKE, 1, FAKE, None)
    assert st == dar.DAR_E_ARG


@no_gpu
def test_decode_rejects():
    s = S()
    need = dar.dar_decode_workspace_bytes(s, 64)
    empty = cache_struct(cap=64, length=0)
    st = dar.lib.dar_attn_decode(ctypes.byref(s), ctypes.byref(empty), FAKE, FAKE, None, FAKE,
                                 FAKE, need, None)
    assert st == dar.DAR_E_ARG  # nothing cached yet
    c = cache_struct(cap=64, length=10)
    st = dar.lib.dar_attn_decode(ctypes.byref(s), ctypes.byref(c), FAKE, FAKE, None, FAKE, FAKE,
                                 need - 4, None)
    assert st == dar.DAR_E_WORKSPACE
    s3 = S(Hq=6, Hkv=2)
    st = dar.lib.dar_attn_decode(ctypes.byref(s3), ctypes.byref(c), FAKE, FAKE, None, FAKE, FAKE,
                                 1 << 30, None)
    assert st == dar.DAR_E_UNSUPPORTED


def test_noalloc_decode_sizes():
    assert dar.dar_decode_noalloc_max_bytes() == 16 << 20
    # decode1b: one workgroup per (batch, KV head) finishes the output, no records
    s = dar.make_shape(32, 32, 8, 64, 16, 512, torch.bfloat16)
    assert dar.dar_decode_noalloc_bytes(s, 32768) == 0
    # few heads and a long cache: P parts, one record of 2 + d_down + d floats per head
    s = dar.make_shape(1, 8, 2, 64, 16, 32, torch.bfloat16)
    n = dar.dar_decode_noalloc_bytes(s, 20000)
    assert n > 0 and n % (8 * (2 + 16 + 64) * 4) == 0
    assert n <= dar.dar_decode_workspace_bytes(s, 20000)
    assert dar.dar_decode_noalloc_bytes(S(Hq=12, Hkv=4), 100) == 0  # group of 3: unsupported


@no_gpu
def test_noalloc_decode_rejects_beyond_its_array():
    """A call that would need more partial records than the fixed array holds
    is refused before anything touches HIP."""
    s = dar.make_shape(8, 64, 8, 256, 64, 16, torch.float32)
    need = dar.dar_decode_noalloc_bytes(s, 100000)
    assert need > dar.dar_decode_noalloc_max_bytes()
    c = cache_struct(cap=100000, length=100000)
    st = dar.lib.dar_attn_decode_noalloc(ctypes.byref(s), ctypes.byref(c), FAKE, FAKE, None, FAKE,
                                         None)
    assert st == dar.DAR_E_WORKSPACE
    c0 = cache_struct(cap=64, length=0)  # nothing cached yet
    st = dar.lib.dar_attn_decode_noalloc(ctypes.byref(S()), ctypes.byref(c0), FAKE, FAKE, None,
                                         FAKE, None)
    assert st == dar.DAR_E_ARG


def test_python_binding_names_match_abi():
    for n in declared_functions():
        assert hasattr(dar, n), n


def expected_backward_ws(B, Hq, Hkv, T, d, dd):
    """The larger of the two kernel families' layouts (every part 256-byte
    aligned, token counts padded to a multiple of 64):
      lse and delta per row (fp32);
      two per-row operand arrays (q W_up^T, dO W_up^T) and two per-key ones
      (the latents): fp32 [dd] each for the vector-ALU kernels; bf16 [dd] plus
      a transposed 32-row block padded to 32 latent rows for the matrix-core
      kernels, which also keep 16 bf16 row constants per row;
      two d_down-wide fp32 sums per row and two per key;
      weight partials: over min(128, ceil(rows/256)) row chunks (vector ALU) or
      one per 128-row workgroup (matrix core)."""
    al = lambda x: (x + 255) // 256 * 256
    Tr = (T + 63) // 64 * 64
    rows, toks = B * Hq * Tr, B * Hkv * Tr
    G = Hq // Hkv

    def layout(mfma):
        opw = (dd + 32) * 2 if mfma else dd * 4
        if mfma:
            nblk = (T + 127) // 128
            nchunk = max(B * nblk, B * G * nblk)
        else:
            nch = lambda r: min(128, max(1, (r + 255) // 256))
            nchunk = max(nch(B * T), nch(B * G * T))
        return (2 * al(rows * 4) + 2 * al(rows * opw) + (al(rows * 32) if mfma else 0)
                + 2 * al(rows * dd * 4) + 2 * al(toks * opw) + 2 * al(toks * dd * 4)
                + al(2 * Hkv * nchunk * d * dd * 4))
    return max(layout(False), layout(True))


def test_backward_workspace_size():
    for kw, T in (({}, 100), ({"Hq": 8, "Hkv": 2}, 3000), ({"d": 128, "dd": 32}, 1)):
        s = S(**kw)
        assert dar.dar_prefill_backward_workspace_bytes(s, T) == expected_backward_ws(
            s.B, s.Hq, s.Hkv, T, s.d, s.d_down)
    assert dar.dar_prefill_backward_workspace_bytes(S(Hq=3), 64) == 0
    assert dar.dar_prefill_backward_workspace_bytes(S(), 0) == 0


def call_backward(shape, T=16, wu=None, dwu=None, ws=FAKE, ws_bytes=1 << 30, **kw):
    args = dict(q=FAKE, k=FAKE, v=FAKE, wd=FAKE, o=FAKE, lse=FAKE, dout=FAKE, dq=FAKE, dk=FAKE,
                dv=FAKE, dwd=FAKE)
    args.update(kw)
    return dar.lib.dar_attn_prefill_backward(
        ctypes.byref(shape), T, args["q"], args["k"], args["v"], args["wd"], wu, args["o"],
        args["lse"], args["dout"], args["dq"], args["dk"], args["dv"], args["dwd"], dwu, ws,
        ws_bytes, None)


@no_gpu
@pytest.mark.parametrize("kw,shape_kw,expect", [
    ({}, {"Hq": 3}, dar.DAR_E_ARG),
    ({"T": 0}, {}, dar.DAR_E_ARG),
    ({"dout": None}, {}, dar.DAR_E_ARG),
    ({"lse": None}, {}, dar.DAR_E_ARG),
    ({"o": MISALIGNED}, {}, dar.DAR_E_ARG),
    ({"dwd": None}, {}, dar.DAR_E_ARG),
    ({"wu": FAKE}, {}, dar.DAR_E_ARG),             # untied needs dw_up
    ({"dwu": FAKE}, {}, dar.DAR_E_ARG),            # tied must not pass dw_up
    ({"wu": FAKE, "dwu": MISALIGNED}, {}, dar.DAR_E_ARG),
    ({"ws": None, "ws_bytes": 0}, {}, dar.DAR_E_WORKSPACE),
    ({"ws_bytes": 16}, {}, dar.DAR_E_WORKSPACE),
    ({}, {"d": 512, "dd": 16}, dar.DAR_E_UNSUPPORTED),
])
def test_backward_rejects(kw, shape_kw, expect):
    assert call_backward(S(**shape_kw), **kw) == expect



def test_chunk_workspace_size():
    """Context copy of K and V (ring tokens from max(0, len - w), then the n new
    ones) followed, on the matrix-core shapes (latents read in place), by the
    two block-norm arrays of ceil((len + n) / 32) blocks a head, else by the
    prefill workspace of len + n positions."""
    al = lambda x: (x + 255) // 256 * 256
    for (B, Hq, Hkv, d, dd, w, dt, es), (L, n) in [((2, 4, 2, 64, 16, 8, torch.bfloat16, 2), (100, 7)),
                                                   ((2, 4, 2, 64, 16, 8, torch.bfloat16, 2), (3, 50)),
                                                   ((1, 2, 2, 128, 32, 40, torch.bfloat16, 2), (300, 1)),
                                                   ((1, 2, 2, 64, 8, 4, torch.bfloat16, 2), (30, 9)),
                                                   ((1, 2, 2, 16, 4, 0, torch.float32, 4), (40, 9))]:
        s = dar.make_shape(B, Hq, Hkv, d, dd, w, dt)
        kv0 = max(0, L - w)
        ctx = al(B * Hkv * (L + n - kv0) * d * es)
        if dt == torch.bfloat16 and d in (64, 128) and dd in (16, 32):
            want = 2 * ctx + 2 * al(B * Hkv * ((L + n + 31) // 32) * 4)
        else:
            want = 2 * ctx + expected_prefill_ws(B, Hkv, L + n, dd, w, es)
        assert dar.dar_prefill_chunk_workspace_bytes(s, L, n) == want
    s = S()
    assert dar.dar_prefill_chunk_workspace_bytes(s, 10, 0) == 0    # n >= 1
    assert dar.dar_prefill_chunk_workspace_bytes(s, -1, 4) == 0    # len >= 0
    assert dar.dar_prefill_chunk_workspace_bytes(S(Hq=3), 4, 4) == 0


def call_chunk(shape, c, n=5, q=FAKE, k=FAKE, v=FAKE, wd=FAKE, wu=None, o=FAKE, lse=None,
               ws=FAKE, ws_bytes=1 << 30):
    return dar.lib.dar_attn_prefill_chunk(ctypes.byref(shape), ctypes.byref(c), n, q, k, v, wd,
                                          wu, o, lse, ws, ws_bytes, None)


@no_gpu
def test_chunk_rejects_before_any_launch():
    s = S()
    c = cache_struct(cap=64, length=60)
    assert call_chunk(s, c, n=5) == dar.DAR_E_CAPACITY and c.len == 60
    assert call_chunk(s, c, n=0) == dar.DAR_E_ARG and c.len == 60
    assert call_chunk(s, c, n=2, q=None) == dar.DAR_E_ARG and c.len == 60
    assert call_chunk(s, c, n=2, k=MISALIGNED) == dar.DAR_E_ARG and c.len == 60
    assert call_chunk(s, c, n=2, wu=MISALIGNED) == dar.DAR_E_ARG and c.len == 60
    assert call_chunk(s, c, n=2, lse=MISALIGNED) == dar.DAR_E_ARG and c.len == 60
    assert call_chunk(s, c, n=2, ws_bytes=64) == dar.DAR_E_WORKSPACE and c.len == 60
    assert call_chunk(s, c, n=2, ws=None, ws_bytes=0) == dar.DAR_E_WORKSPACE and c.len == 60
    assert call_chunk(S(Hq=3), c, n=2) == dar.DAR_E_ARG and c.len == 60
    c2 = cache_struct(win=None)  # a ring is required when w > 0
    assert call_chunk(s, c2, n=2) == dar.DAR_E_ARG and c2.len == 0
    # bf16 rows of an odd number of elements cannot be copied in 4-byte words
    assert call_chunk(S(d=63, dd=16), cache_struct(), n=2) == dar.DAR_E_UNSUPPORTED


def test_chunk_rope_workspace_size():
    """Context rows from the window's oldest position rounded down to 32 (len
    with w = 0), rotated chunk queries, rotated context keys, lifted distant
    keys and values (positions < len + n - w), block norms; 256-byte aligned."""
    al = lambda x: (x + 255) // 256 * 256
    for (B, Hq, Hkv, d, dd, w), (L, n) in [((2, 4, 2, 64, 16, 40), (100, 7)),
                                           ((2, 4, 2, 64, 16, 40), (3, 50)),
                                           ((1, 8, 2, 128, 32, 0), (70, 9))]:
        s = dar.make_shape(B, Hq, Hkv, d, dd, w, torch.bfloat16)
        kv0 = (max(0, L - w) // 32) * 32 if w > 0 else L
        Tc, T = L + n - kv0, L + n
        Td = max(T - w, 0)
        ctx = al(B * Hkv * Tc * d * 2)
        want = (3 * ctx + al(B * Hq * n * d * 2) + 2 * al(B * Hkv * Td * d * 2)
                + al(B * Hkv * ((T + 31) // 32) * 4) + al(B * Hkv * ((Td + 31) // 32 + 1) * 4))
        assert dar.dar_prefill_chunk_rope_workspace_bytes(s, L, n) == want
    assert dar.dar_prefill_chunk_rope_workspace_bytes(S(), 10, 0) == 0
    assert dar.dar_prefill_chunk_rope_workspace_bytes(S(), -1, 4) == 0


@no_gpu
def test_chunk_rope_rejects_before_any_launch():
    def call(shape, c, n=2, r=16, n_pos=128, table=FAKE, q=FAKE, ws_bytes=1 << 30, null_rope=False):
        rs = dar.DarRopeStruct(r, n_pos, table)
        return dar.lib.dar_attn_prefill_chunk_rope(
            ctypes.byref(shape), ctypes.byref(c), None if null_rope else ctypes.byref(rs), n, q, FAKE,
            FAKE, FAKE, None, FAKE, None, FAKE, ws_bytes, None)
    s = S()
    c = cache_struct(cap=64, length=60)
    assert call(s, c, n=5) == dar.DAR_E_CAPACITY and c.len == 60
    assert call(s, c, null_rope=True) == dar.DAR_E_ARG and c.len == 60
    assert call(s, c, n_pos=61) == dar.DAR_E_ARG and c.len == 60          # past the table
    assert call(s, c, r=5) == dar.DAR_E_ARG and c.len == 60
    assert call(s, c, table=None) == dar.DAR_E_ARG and c.len == 60
    assert call(s, c, q=MISALIGNED) == dar.DAR_E_ARG and c.len == 60
    assert call(s, c, ws_bytes=64) == dar.DAR_E_WORKSPACE and c.len == 60
    assert call(s, c, r=8) == dar.DAR_E_UNSUPPORTED and c.len == 60       # r % 16
    assert call(S(dtype=torch.float32), c) == dar.DAR_E_UNSUPPORTED and c.len == 60
    assert call(S(d=80, dd=20), c) == dar.DAR_E_UNSUPPORTED and c.len == 60


def test_rope_workspace_size():
    """Rotated queries and keys, lifted distant keys and values (positions
    < T - w), block norms of both key arrays; 256-byte aligned parts."""
    al = lambda x: (x + 255) // 256 * 256
    for (B, Hq, Hkv, d, dd, w, dt, es), T in [((2, 4, 2, 64, 16, 8, torch.bfloat16, 2), 100),
                                              ((2, 4, 2, 64, 16, 8, torch.bfloat16, 2), 5),
                                              ((1, 2, 1, 16, 4, 0, torch.float32, 4), 33)]:
        s = dar.make_shape(B, Hq, Hkv, d, dd, w, dt)
        Td = max(T - w, 0)
        want = (al(B * Hq * T * d * es) + al(B * Hkv * T * d * es) + 2 * al(B * Hkv * Td * d * es)
                + al(B * Hkv * ((T + 31) // 32) * 4) + al(B * Hkv * ((Td + 31) // 32) * 4) + 256)
        assert dar.dar_prefill_rope_workspace_bytes(s, T) == want
    assert dar.dar_prefill_rope_workspace_bytes(S(), 0) == 0
    assert dar.dar_prefill_rope_workspace_bytes(S(Hq=3), 8) == 0


def call_rope(shape, T=16, pos0=0, r=64, n_pos=64, table=FAKE, q=FAKE, k=FAKE, v=FAKE, wd=FAKE,
              wu=None, o=FAKE, lse=None, ws=FAKE, ws_bytes=1 << 30, null_rope=False):
    rs = dar.DarRopeStruct(r, n_pos, table)
    return dar.lib.dar_attn_prefill_rope(ctypes.byref(shape), T, pos0,
                                         None if null_rope else ctypes.byref(rs), q, k, v, wd, wu,
                                         o, lse, ws, ws_bytes, None)


@no_gpu
def test_rope_rejects_before_any_launch():
    s = S()
    assert call_rope(s, null_rope=True) == dar.DAR_E_ARG
    assert call_rope(s, r=63) == dar.DAR_E_ARG            # odd rotary dimension
    assert call_rope(s, r=66) == dar.DAR_E_ARG            # wider than d
    assert call_rope(s, r=-2) == dar.DAR_E_ARG
    assert call_rope(s, table=None) == dar.DAR_E_ARG      # r > 0 needs the table
    assert call_rope(s, table=MISALIGNED) == dar.DAR_E_ARG
    assert call_rope(s, T=60, pos0=5, n_pos=64) == dar.DAR_E_ARG   # positions past the table
    assert call_rope(s, pos0=-1) == dar.DAR_E_ARG
    assert call_rope(s, T=0) == dar.DAR_E_ARG
    assert call_rope(s, q=None) == dar.DAR_E_ARG
    assert call_rope(s, wu=MISALIGNED) == dar.DAR_E_ARG
    assert call_rope(s, ws_bytes=64) == dar.DAR_E_WORKSPACE
    assert call_rope(s, ws=None, ws_bytes=0) == dar.DAR_E_WORKSPACE
    assert call_rope(S(Hq=3)) == dar.DAR_E_ARG
    st = dar.lib.dar_rope_table
    assert st(63, 10000.0, 8, FAKE, None) == dar.DAR_E_ARG
    assert st(0, 10000.0, 8, FAKE, None) == dar.DAR_E_ARG
    assert st(64, 0.0, 8, FAKE, None) == dar.DAR_E_ARG
    assert st(64, 10000.0, 0, FAKE, None) == dar.DAR_E_ARG
    assert st(64, 10000.0, 8, None, None) == dar.DAR_E_ARG
    assert st(64, 10000.0, 70000, FAKE, None) == dar.DAR_E_UNSUPPORTED


@no_gpu
def test_decode_rope_rejects_before_any_launch():
    s = S()
    def call(c, r=64, n_pos=64, table=FAKE, q=FAKE, ws_bytes=1 << 30, null_rope=False):
        rs = dar.DarRopeStruct(r, n_pos, table)
        return dar.lib.dar_attn_decode_rope(ctypes.byref(s), ctypes.byref(c),
                                            None if null_rope else ctypes.byref(rs), q, FAKE, None,
                                            FAKE, FAKE, ws_bytes, None)
    assert call(cache_struct(cap=64, length=10), null_rope=True) == dar.DAR_E_ARG
    assert call(cache_struct(cap=64, length=0)) == dar.DAR_E_ARG        # empty cache
    assert call(cache_struct(cap=100, length=70), n_pos=64) == dar.DAR_E_ARG  # past the table
    assert call(cache_struct(cap=64, length=10), r=5) == dar.DAR_E_ARG
    assert call(cache_struct(cap=64, length=10), table=None) == dar.DAR_E_ARG
    assert call(cache_struct(cap=64, length=10), q=MISALIGNED) == dar.DAR_E_ARG
    assert call(cache_struct(cap=64, length=10), ws_bytes=8) == dar.DAR_E_WORKSPACE


@no_gpu
def test_shared_latent_rejects_before_any_launch():
    s = S()
    pf = lambda T=16, c=FAKE, uv=FAKE, ws_bytes=1 << 30: dar.lib.dar_attn_prefill_shared(
        ctypes.byref(s), T, FAKE, FAKE, FAKE, c, FAKE, uv, FAKE, None, FAKE, ws_bytes, None)
    assert pf(c=None) == dar.DAR_E_ARG
    assert pf(uv=MISALIGNED) == dar.DAR_E_ARG
    assert pf(T=0) == dar.DAR_E_ARG
    assert pf(ws_bytes=16) == dar.DAR_E_WORKSPACE
    c = cache_struct(cap=64, length=60)
    ap = lambda n=2, cn=FAKE: dar.lib.dar_cache_append_shared(ctypes.byref(s), ctypes.byref(c),
                                                             FAKE, FAKE, cn, n, None)
    assert ap(n=5) == dar.DAR_E_CAPACITY and c.len == 60
    assert ap(cn=None) == dar.DAR_E_ARG and c.len == 60
    assert ap(n=0) == dar.DAR_E_ARG and c.len == 60
    dc = lambda cc, uk=FAKE, ws_bytes=1 << 30: dar.lib.dar_attn_decode_shared(
        ctypes.byref(s), ctypes.byref(cc), FAKE, uk, FAKE, FAKE, FAKE, ws_bytes, None)
    assert dc(cache_struct(cap=64, length=0)) == dar.DAR_E_ARG
    assert dc(cache_struct(cap=64, length=10), uk=None) == dar.DAR_E_ARG
    assert dc(cache_struct(cap=64, length=10), ws_bytes=8) == dar.DAR_E_WORKSPACE


@no_gpu
def test_paged_rejects_before_any_launch():
    s = S()
    def pc(ps=64, maxb=4, n_pages=8, pool=FAKE, bt=FAKE, lens=FAKE, win=FAKE):
        return dar.DarPagedCacheStruct(win.value if win else None, win.value if win else None,
                                       pool.value if pool else None, FAKE.value,
                                       bt.value if bt else None, lens.value if lens else None,
                                       ps, maxb, n_pages)
    ap = lambda c, k=FAKE: dar.lib.dar_cache_append_paged(ctypes.byref(s), ctypes.byref(c), k, FAKE,
                                                          FAKE, None)
    dc = lambda c, ws_bytes=1 << 30, shape=s: dar.lib.dar_attn_decode_paged(
        ctypes.byref(shape), ctypes.byref(c), FAKE, FAKE, None, FAKE, FAKE, ws_bytes, None)
    assert ap(pc(ps=48)) == dar.DAR_E_ARG          # page size not a power of two
    assert ap(pc(ps=96)) == dar.DAR_E_ARG
    assert ap(pc(ps=0)) == dar.DAR_E_ARG
    assert ap(pc(maxb=0)) == dar.DAR_E_ARG
    assert ap(pc(n_pages=0)) == dar.DAR_E_ARG
    assert ap(pc(pool=None)) == dar.DAR_E_ARG
    assert ap(pc(bt=None)) == dar.DAR_E_ARG
    assert ap(pc(lens=None)) == dar.DAR_E_ARG
    assert ap(pc(lens=ctypes.c_void_p((1 << 20) + 2))) == dar.DAR_E_ARG   # int array misaligned
    assert ap(pc(win=None)) == dar.DAR_E_ARG       # a ring is required when w > 0
    assert ap(pc(), k=MISALIGNED) == dar.DAR_E_ARG
    assert dc(pc(), ws_bytes=8) == dar.DAR_E_WORKSPACE
    assert dc(pc(), shape=S(dtype=torch.float32)) == dar.DAR_E_UNSUPPORTED   # matrix-core shapes only
    assert dc(pc(), shape=S(d=80, dd=16)) == dar.DAR_E_UNSUPPORTED


@no_gpu
def test_paged_rope_rejects_before_any_launch():
    """Capacity 4 pages of 64 = 256 positions."""
    c = dar.DarPagedCacheStruct(FAKE.value, FAKE.value, FAKE.value, FAKE.value, FAKE.value,
                                FAKE.value, 64, 4, 8)
    def call(r=64, n_pos=256, table=FAKE, shape=None, null_rope=False, ws_bytes=1 << 30):
        rs = dar.DarRopeStruct(r, n_pos, table)
        return dar.lib.dar_attn_decode_paged_rope(ctypes.byref(shape or S()), ctypes.byref(c),
                                                  None if null_rope else ctypes.byref(rs), FAKE,
                                                  FAKE, None, FAKE, FAKE, ws_bytes, None)
    assert call(null_rope=True) == dar.DAR_E_ARG
    assert call(n_pos=255) == dar.DAR_E_ARG        # a reachable position past the table
    assert call(r=5) == dar.DAR_E_ARG
    assert call(r=-2) == dar.DAR_E_ARG
    assert call(r=66) == dar.DAR_E_ARG             # above d
    assert call(table=None) == dar.DAR_E_ARG
    assert call(r=24) == dar.DAR_E_UNSUPPORTED
    assert call(shape=S(d=128, dd=48)) == dar.DAR_E_UNSUPPORTED
    assert call(ws_bytes=8) == dar.DAR_E_WORKSPACE
    assert call(r=0, table=None, ws_bytes=8) == dar.DAR_E_WORKSPACE   # r = 0 reads no table


def test_chunk_paged_workspace_size():
    """Context rows of every sequence (w + n rows a head) for K and V, then two
    block-norm arrays covering a whole sequence's capacity."""
    al = lambda x: (x + 255) // 256 * 256
    for (B, Hkv, d, dd, w), (cap, n) in [((4, 2, 64, 16, 32), (4096, 256)),
                                          ((3, 8, 128, 32, 0), (100, 1))]:
        s = dar.make_shape(B, Hkv * 4, Hkv, d, dd, w, torch.bfloat16)
        want = 2 * al(B * Hkv * (w + n) * d * 2) + 2 * al(B * Hkv * ((cap + 31) // 32) * 4)
        assert dar.dar_prefill_chunk_paged_workspace_bytes(s, cap, n) == want
    assert dar.dar_prefill_chunk_paged_workspace_bytes(S(), 64, 0) == 0
    assert dar.dar_prefill_chunk_paged_workspace_bytes(S(), 0, 4) == 0


@no_gpu
def test_chunk_paged_rejects_before_any_launch():
    def pc(ps=64, maxb=4, n_pages=8, bt=FAKE, lens=FAKE, win=FAKE):
        return dar.DarPagedCacheStruct(win.value if win else None, win.value if win else None,
                                       FAKE.value, FAKE.value, bt.value if bt else None,
                                       lens.value if lens else None, ps, maxb, n_pages)
    def call(c=None, shape=None, n=8, n_new=None, q=FAKE, wu=None, lse=None, ws_bytes=1 << 30):
        shape = shape or S()
        c = c or pc()
        return dar.lib.dar_attn_prefill_chunk_paged(ctypes.byref(shape), ctypes.byref(c), n, n_new, q,
                                                    FAKE, FAKE, FAKE, wu, FAKE, lse, FAKE, ws_bytes,
                                                    None)
    assert call(n=0) == dar.DAR_E_ARG
    assert call(c=pc(ps=48)) == dar.DAR_E_ARG
    assert call(c=pc(bt=None)) == dar.DAR_E_ARG
    assert call(c=pc(lens=None)) == dar.DAR_E_ARG
    assert call(c=pc(win=None)) == dar.DAR_E_ARG
    assert call(q=None) == dar.DAR_E_ARG
    assert call(q=MISALIGNED) == dar.DAR_E_ARG
    assert call(wu=MISALIGNED) == dar.DAR_E_ARG
    assert call(lse=MISALIGNED) == dar.DAR_E_ARG
    assert call(n_new=ctypes.c_void_p((1 << 20) + 2)) == dar.DAR_E_ARG   # int array misaligned
    assert call(ws_bytes=64) == dar.DAR_E_WORKSPACE
    assert call(shape=S(dtype=torch.float32)) == dar.DAR_E_UNSUPPORTED   # matrix-core shapes only
    assert call(shape=S(d=64, dd=8)) == dar.DAR_E_UNSUPPORTED
    assert call(shape=S(Hq=3)) == dar.DAR_E_ARG


def test_rope_backward_workspace_size():
    """Rotated queries and keys, lifted distant keys and values (bf16), two
    row constants, the fp32 row, window-key and distant-key gradients and the
    weight-gradient shares (one per 32 keys of a sequence)."""
    al = lambda x: (x + 255) // 256 * 256
    for (B, Hq, Hkv, d, dd, w), T in [((2, 4, 2, 64, 16, 32), 300), ((1, 8, 2, 128, 32, 500), 400)]:
        s = dar.make_shape(B, Hq, Hkv, d, dd, w, torch.bfloat16)
        Td = max(T - w, 0)
        Tr = (T + 63) // 64 * 64
        nchunk = B * ((T + 31) // 32)
        want = (al(B * Hq * T * d * 2) + al(B * Hkv * T * d * 2) + 2 * al(B * Hkv * Td * d * 2)
                + 2 * al(B * Hq * Tr * 4) + al(B * Hq * T * d * 4) + 2 * al(B * Hkv * T * d * 4)
                + 2 * al(B * Hkv * Td * d * 4) + al(2 * Hkv * nchunk * d * dd * 4))
        assert dar.dar_prefill_rope_backward_workspace_bytes(s, T) == want
    assert dar.dar_prefill_rope_backward_workspace_bytes(S(), 0) == 0
    assert dar.dar_prefill_rope_backward_workspace_bytes(S(Hq=3), 10) == 0


@no_gpu
def test_rope_backward_rejects_before_any_launch():
    rs = dar.DarRopeStruct(16, 64, FAKE.value)
    def call(shape=None, T=32, pos0=0, rope=rs, q=FAKE, wu=None, dwu=None, lse=FAKE,
             ws_bytes=1 << 30):
        shape = shape or S()
        return dar.lib.dar_attn_prefill_rope_backward(
            ctypes.byref(shape), T, pos0, ctypes.byref(rope) if rope is not None else None, q, FAKE,
            FAKE, FAKE, wu, FAKE, lse, FAKE, FAKE, FAKE, FAKE, FAKE, dwu, FAKE, ws_bytes, None)
    assert call(T=0) == dar.DAR_E_ARG
    assert call(pos0=-1) == dar.DAR_E_ARG
    assert call(pos0=40) == dar.DAR_E_ARG                          # pos0 + T past the table
    assert call(rope=dar.DarRopeStruct(15, 64, FAKE.value)) == dar.DAR_E_ARG   # odd rotary dim
    assert call(rope=dar.DarRopeStruct(80, 64, FAKE.value)) == dar.DAR_E_ARG   # r > d
    assert call(q=None) == dar.DAR_E_ARG
    assert call(lse=MISALIGNED) == dar.DAR_E_ARG
    assert call(wu=FAKE) == dar.DAR_E_ARG                          # untied needs dw_up
    assert call(dwu=FAKE) == dar.DAR_E_ARG                         # tied takes no dw_up
    assert call(ws_bytes=64) == dar.DAR_E_WORKSPACE
    assert call(shape=S(dtype=torch.float32)) == dar.DAR_E_UNSUPPORTED
    assert call(shape=S(d=80, dd=16)) == dar.DAR_E_UNSUPPORTED
    assert call(shape=S(d=128, dd=96)) == dar.DAR_E_UNSUPPORTED


@no_gpu
def test_ragged_prefill_rejects_before_any_launch():
    s = S()
    call = lambda T=16, lens=FAKE, q=FAKE, ws_bytes=1 << 30: dar.lib.dar_attn_prefill_ragged(
        ctypes.byref(s), T, lens, q, FAKE, FAKE, FAKE, None, FAKE, None, FAKE, ws_bytes, None)
    assert call(lens=None) == dar.DAR_E_ARG
    assert call(lens=ctypes.c_void_p((1 << 20) + 2)) == dar.DAR_E_ARG
    assert call(T=0) == dar.DAR_E_ARG
    assert call(q=MISALIGNED) == dar.DAR_E_ARG
    assert call(ws_bytes=16) == dar.DAR_E_WORKSPACE


def test_ragged_prefill_binding_checks_lengths():
    """The binding rejects lengths that are not an int32 tensor of shape (B,)
    on the device, before any call into the library."""
    q = torch.zeros(2, 2, 8, 64, dtype=torch.bfloat16)
    k = torch.zeros(2, 1, 8, 64, dtype=torch.bfloat16)
    wd = torch.zeros(1, 64, 16, dtype=torch.bfloat16)
    for lens in (torch.tensor([8, 3], dtype=torch.int64), torch.tensor([8], dtype=torch.int32),
                 torch.tensor([8, 3], dtype=torch.int32)):   # the last one is on the host
        with pytest.raises(ValueError):
            dar.dar_attn_prefill_ragged(q, k, k, wd, None, 4, lens)


def test_bench_refuses_several_gpus():
    """bench.py measures one GPU: --gpus 2 exits with status 2 and says so."""
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    r = subprocess.run([sys.executable, os.path.join(root, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=300)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
