"""Binding of libdar_k0.so (include/dar_k0.h): the machine microbenchmarks
that fix the ceilings the DAR kernels are measured against (bf16 matrix-core
rate, v_exp_f32 rate, their overlap, streaming HBM, shader clock under load).
Measurement only; the attention path does not use it."""
from __future__ import annotations

import ctypes
import os

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
K0_LIB_PATH = os.path.join(_PKG, "libdar_k0.so")


class DarK0Result(ctypes.Structure):
    _fields_ = [("n_cu", ctypes.c_int),
                ("mfma_bf16_tflops", ctypes.c_double * 3),
                ("mfma_clock_mhz", ctypes.c_double),
                ("exp_lanes_per_clk_cu", ctypes.c_double),
                ("exp_per_s", ctypes.c_double),
                ("exp_clock_mhz", ctypes.c_double),
                ("mix_cycles_per_iter", ctypes.c_double),
                ("mfma_only_cycles_per_iter", ctypes.c_double),
                ("exp_only_cycles_per_iter", ctypes.c_double),
                ("fma_only_cycles_per_iter", ctypes.c_double),
                ("mix_fma_cycles_per_iter", ctypes.c_double),
                ("hbm_read_gbs", ctypes.c_double),
                ("hbm_write_gbs", ctypes.c_double)]


def _load():
    if not os.path.exists(K0_LIB_PATH):
        raise ImportError("libdar_k0.so is not built; run `python paper_2606_18587_amd/build.py`")
    lib = ctypes.CDLL(K0_LIB_PATH)
    lib.dar_k0_measure.restype = ctypes.c_int
    lib.dar_k0_measure.argtypes = [ctypes.c_void_p, ctypes.c_size_t,
                                   ctypes.POINTER(DarK0Result), ctypes.c_void_p]
    return lib


def measure(device="cuda", buf_bytes=2 << 30) -> dict:
    """Run every microbenchmark once on `device` (a 2 GiB scratch buffer,
    larger than L2 and the Infinity Cache) and return the figures."""
    lib = _load()
    buf = torch.empty(buf_bytes, dtype=torch.uint8, device=device)
    r = DarK0Result()
    st = lib.dar_k0_measure(ctypes.c_void_p(buf.data_ptr()), buf_bytes, ctypes.byref(r),
                            ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream))
    del buf
    if st != 0:
        raise RuntimeError("dar_k0_measure failed (status %d)" % st)
    return {
        "n_cu": r.n_cu,
        "mfma_bf16_tflops": {"1_wave_per_simd": round(r.mfma_bf16_tflops[0], 1),
                             "2_waves_per_simd": round(r.mfma_bf16_tflops[1], 1),
                             "4_waves_per_simd": round(r.mfma_bf16_tflops[2], 1)},
        "mfma_clock_mhz": round(r.mfma_clock_mhz, 1),
        "exp_lanes_per_clk_cu": round(r.exp_lanes_per_clk_cu, 2),
        "exp_per_s": r.exp_per_s,
        "exp_clock_mhz": round(r.exp_clock_mhz, 1),
        "mix_8mfma_16exp_cycles": round(r.mix_cycles_per_iter, 1),
        "mfma8_only_cycles": round(r.mfma_only_cycles_per_iter, 1),
        "exp16_only_cycles": round(r.exp_only_cycles_per_iter, 1),
        "fma16_only_cycles": round(r.fma_only_cycles_per_iter, 1),
        "mix_8mfma_16fma_cycles": round(r.mix_fma_cycles_per_iter, 1),
        "hbm_read_gbs": round(r.hbm_read_gbs, 1),
        "hbm_write_gbs": round(r.hbm_write_gbs, 1),
    }


if __name__ == "__main__":
    import json

    print(json.dumps({"k0": measure()}), flush=True)
