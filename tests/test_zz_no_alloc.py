"""dar_attn_decode_noalloc (through the C ABI): the decode entry point that
takes no workspace and allocates nothing, its partial records held in a fixed
device array inside the library. Checked against dar_attn_decode on the same
cache and query, for two calls in a row, the second with a smaller input
(the array keeps the first call's records: the second must not read them).
Both entry points run the same kernels, so the outputs must be bit-identical
(stricter than the 1e-4 / 2e-2 tolerance of the parity tests)."""
import numpy as np
import pytest
import torch

import dar_inputs as di
from tests.dev import to_dev

pytestmark = pytest.mark.gpu

dar = pytest.importorskip("paper_2606_18587_amd")

TDT = {"bf16": torch.bfloat16, "f32": torch.float32}


def make_cache(wl, L):
    pre = di.make_decode_prefix(wl, L)
    c = dar.DarCache(wl.B, wl.Hkv, wl.d, wl.dd, wl.w, L, TDT[wl.dtype])
    wd = to_dev(pre["wd"])
    dar.dar_cache_append(c, to_dev(pre["k"]), to_dev(pre["v"]), wd, Hq=wl.Hq)
    q = to_dev(di.make_decode_step(wl, 0)["q"])
    return c, q, wd


def both(wl, L):
    c, q, wd = make_cache(wl, L)
    shape = dar.make_shape(wl.B, wl.Hq, wl.Hkv, wl.d, wl.dd, wl.w, TDT[wl.dtype])
    used = dar.dar_decode_noalloc_bytes(shape, L)
    print("[noalloc] %s B%d Hq%d Hkv%d d%d dd%d w%d L%d: %d bytes of the fixed array" % (
        wl.dtype, wl.B, wl.Hq, wl.Hkv, wl.d, wl.dd, wl.w, L, used), flush=True)
    o_na = torch.full_like(q, float("nan"))
    dar.dar_attn_decode_noalloc(c, q, wd, o=o_na)
    o_ws = torch.full_like(q, float("nan"))
    dar.dar_attn_decode(c, q, wd, o=o_ws)
    torch.cuda.synchronize()
    bits = torch.int16 if q.dtype == torch.bfloat16 else torch.int32
    assert torch.isfinite(o_na.float()).all()
    assert torch.equal(o_na.view(bits), o_ws.view(bits))
    return used


@pytest.mark.parametrize("first,second", [
    # matrix-core path split over several workgroups per (batch, KV head): records used
    ((di.Workload("na_big", 60, 1, 8, 2, 0, 64, 16, 32, "bf16"), 20000),
     (di.Workload("na_small", 61, 1, 4, 1, 0, 64, 16, 32, "bf16"), 3000)),
    ((di.Workload("na_d128", 62, 1, 8, 2, 0, 128, 32, 100, "bf16"), 9000),
     (di.Workload("na_d128s", 63, 1, 2, 2, 0, 128, 32, 100, "bf16"), 700)),
    # generic path (fp32): split records and the combine kernel
    ((di.Workload("na_f32", 64, 2, 4, 2, 0, 16, 4, 8, "f32"), 1500),
     (di.Workload("na_f32s", 65, 1, 2, 2, 0, 16, 4, 8, "f32"), 300)),
    # one workgroup per (batch, KV head) finishes the output: no records
    ((di.Workload("na_full", 66, 32, 32, 8, 0, 64, 16, 512, "bf16"), 2000),
     (di.Workload("na_fulls", 67, 8, 32, 8, 0, 64, 16, 512, "bf16"), 600)),
])
def test_noalloc_decode_matches_workspace_decode(first, second):
    used1 = both(*first)
    used2 = both(*second)
    assert used1 <= dar.dar_decode_noalloc_max_bytes()
    assert used2 <= used1
