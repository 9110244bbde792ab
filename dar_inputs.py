"""Seeded synthetic inputs shared by the tests, the benchmark and the smoke check.

This module holds no attention arithmetic: it only draws random numbers,
rounds them to bfloat16 (bit-level round-to-nearest-even) and names the
workload shapes. The oracle and the HIP path both receive exactly the values
produced here.

Workloads (per-head shapes; the paper's models are Pythia-70M/160M/410M
pretraining at sequence length 2048 and OLMo-2-1B fine-tuning, Section 3;
synthetic N(0,1) tensors of the same shapes stand in for their data):

  tiny         B1  Hq2  Hkv2 T64    d16  dd4  w8    fp32
  pythia70m    B8  Hq8  Hkv8 T2048  d64  dd16 w256  bf16
  pythia410m   B4  Hq16 Hkv16 T2048 d64  dd16 w128 / w512  bf16
  decode1b     B32 Hq32 Hkv8 L32768 d64  dd16 w512  bf16, 128 decode steps
  long16k      B1  Hq32 Hkv8 T16384 d128 dd32 w1024 bf16

Down-projections are drawn N(0, 1/d) per KV head, shape [d, d_down]; the
up-projection is tied (W_up = W_down^T) unless a test asks for an untied one,
which is drawn N(0, 1/d_down).
"""
from __future__ import annotations

from dataclasses import dataclass, replace

import numpy as np

SEED_BASE = 260618587

# tensor ids inside one workload's seed space
TID_Q, TID_K, TID_V, TID_WD, TID_WU, TID_DO = 0, 1, 2, 3, 4, 5


@dataclass(frozen=True)
class Workload:
    name: str
    cfg_id: int          # selects the seed space
    B: int
    Hq: int
    Hkv: int
    T: int               # prefill length, or cache length L for decode
    d: int
    dd: int
    w: int
    dtype: str           # "f32" or "bf16"
    kind: str = "prefill"  # "prefill" or "decode"
    steps: int = 0         # decode steps

    def with_(self, **kw) -> "Workload":
        return replace(self, **kw)


WORKLOADS = {
    "tiny": Workload("tiny", 0, 1, 2, 2, 64, 16, 4, 8, "f32"),
    "pythia70m": Workload("pythia70m", 1, 8, 8, 8, 2048, 64, 16, 256, "bf16"),
    "pythia410m_w128": Workload("pythia410m_w128", 2, 4, 16, 16, 2048, 64, 16, 128, "bf16"),
    "pythia410m_w512": Workload("pythia410m_w512", 2, 4, 16, 16, 2048, 64, 16, 512, "bf16"),
    "decode1b": Workload("decode1b", 3, 32, 32, 8, 32768, 64, 16, 512, "bf16",
                         kind="decode", steps=128),
    "long16k": Workload("long16k", 4, 1, 32, 8, 16384, 128, 32, 1024, "bf16"),
}


def seed_for(cfg_id: int, tensor_id: int) -> int:
    return SEED_BASE + 100 * cfg_id + tensor_id


def round_bf16_bits(x: np.ndarray) -> np.ndarray:
    """fp32 -> bfloat16 bit patterns (uint16), round to nearest even."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    flat = x.reshape(-1)
    out = np.empty(flat.shape, np.uint16)
    step = 1 << 24
    for s in range(0, flat.size, step):
        u = flat[s:s + step].view(np.uint32)
        # finite values cannot overflow 32 bits here; NaNs are replaced below
        r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
        out[s:s + step] = r.astype(np.uint16)
    nan = np.isnan(flat)
    if nan.any():
        out[nan] = 0x7FC0
    return out.reshape(x.shape)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


class Tensor:
    """A host tensor in the storage dtype of a workload.

    `store` is what is uploaded (float32 array, or uint16 bf16 bits);
    `f64` is the exact same values widened to float64 for the oracle.
    """

    def __init__(self, values_f32: np.ndarray, dtype: str):
        self.dtype = dtype
        if dtype == "bf16":
            self.store = round_bf16_bits(values_f32)
            self.f64 = bf16_bits_to_f32(self.store).astype(np.float64)
        elif dtype == "f32":
            self.store = np.ascontiguousarray(values_f32, dtype=np.float32)
            self.f64 = self.store.astype(np.float64)
        else:
            raise ValueError(dtype)

    @classmethod
    def from_store(cls, store: np.ndarray, dtype: str) -> "Tensor":
        """Wrap already-rounded storage (uint16 bf16 bits or float32); the
        float64 view is made on demand to keep large caches cheap."""
        t = cls.__new__(cls)
        t.dtype = dtype
        t.store = store
        t._f64 = None
        return t

    @property
    def f64(self) -> np.ndarray:
        if self._f64 is None:
            src = bf16_bits_to_f32(self.store) if self.dtype == "bf16" else self.store
            self._f64 = src.astype(np.float64)
        return self._f64

    @f64.setter
    def f64(self, value):
        self._f64 = value

    def f64_slice(self, idx) -> np.ndarray:
        """float64 values of store[idx] without widening the whole tensor."""
        part = self.store[idx]
        src = bf16_bits_to_f32(part) if self.dtype == "bf16" else part
        return np.asarray(src, dtype=np.float64)

    @property
    def shape(self):
        return self.store.shape


def normal(shape, seed: int, std: float = 1.0) -> np.ndarray:
    g = np.random.Generator(np.random.PCG64(seed))
    return (g.standard_normal(size=shape, dtype=np.float32) * np.float32(std)).astype(np.float32)


def make_prefill_inputs(wl: Workload, untied: bool = False, seed_shift: int = 0,
                        q_scale: float = 1.0) -> dict:
    """Q [B,Hq,T,d], K,V [B,Hkv,T,d], W_down [Hkv,d,dd], optional W_up [Hkv,dd,d]."""
    s = seed_shift
    q = normal((wl.B, wl.Hq, wl.T, wl.d), seed_for(wl.cfg_id, TID_Q) + s) * np.float32(q_scale)
    k = normal((wl.B, wl.Hkv, wl.T, wl.d), seed_for(wl.cfg_id, TID_K) + s)
    v = normal((wl.B, wl.Hkv, wl.T, wl.d), seed_for(wl.cfg_id, TID_V) + s)
    wd = normal((wl.Hkv, wl.d, wl.dd), seed_for(wl.cfg_id, TID_WD) + s, std=1.0 / np.sqrt(wl.d))
    out = {
        "q": Tensor(q, wl.dtype),
        "k": Tensor(k, wl.dtype),
        "v": Tensor(v, wl.dtype),
        "wd": Tensor(wd, wl.dtype),
        "wu": None,
    }
    if untied:
        wu = normal((wl.Hkv, wl.dd, wl.d), seed_for(wl.cfg_id, TID_WU) + s, std=1.0 / np.sqrt(wl.dd))
        out["wu"] = Tensor(wu, wl.dtype)
    return out


def make_backward_inputs(wl: Workload, untied: bool = False, seed_shift: int = 0,
                         q_scale: float = 1.0) -> dict:
    """The prefill inputs plus the incoming gradient dout [B,Hq,T,d] ~ N(0,1)."""
    out = make_prefill_inputs(wl, untied=untied, seed_shift=seed_shift, q_scale=q_scale)
    dout = normal((wl.B, wl.Hq, wl.T, wl.d), seed_for(wl.cfg_id, TID_DO) + seed_shift)
    out["dout"] = Tensor(dout, wl.dtype)
    return out


def make_decode_prefix(wl: Workload, L: int) -> dict:
    """Keys and values [B,Hkv,L,d] of the tokens already in the cache before
    the decode steps, drawn batch by batch from one stream per tensor."""
    out = {}
    for name, tid in (("k", TID_K), ("v", TID_V)):
        g = np.random.Generator(np.random.PCG64(seed_for(wl.cfg_id, tid)))
        parts = []
        for _ in range(wl.B):
            x = g.standard_normal(size=(wl.Hkv, L, wl.d), dtype=np.float32)
            parts.append(round_bf16_bits(x) if wl.dtype == "bf16" else x)
        store = np.stack(parts)
        out[name] = Tensor.from_store(store, wl.dtype)
    wd = normal((wl.Hkv, wl.d, wl.dd), seed_for(wl.cfg_id, TID_WD), std=1.0 / np.sqrt(wl.d))
    out["wd"] = Tensor(wd, wl.dtype)
    out["wu"] = None
    return out


def make_decode_step(wl: Workload, t: int) -> dict:
    """Fresh token k,v [B,Hkv,1,d] and query q [B,Hq,d] for decode step t."""
    base = seed_for(wl.cfg_id, 1000 + 3 * t)
    k = normal((wl.B, wl.Hkv, 1, wl.d), base + 1)
    v = normal((wl.B, wl.Hkv, 1, wl.d), base + 2)
    q = normal((wl.B, wl.Hq, wl.d), base + 0)
    return {"q": Tensor(q, wl.dtype), "k": Tensor(k, wl.dtype), "v": Tensor(v, wl.dtype)}
