"""Build libdar.so (all HIP kernels + the C ABI) for gfx950 with hipcc.

Usage: python paper_2606_18587_amd/build.py [-v]
This file is run as a script (or loaded by path) rather than imported as part
of the package: importing the package needs the library it builds. The
library is built in-tree, next to this file.
"""
from __future__ import annotations

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "libdar.so")
K0_LIB = os.path.join(PKG, "libdar_k0.so")
K0_SOURCE = "k0_microbench.hip"
SOURCES = ["dar_api.hip", "latent.hip", "prefill_valu.hip", "prefill_mfma.hip", "decode.hip",
           "decode_mfma.hip", "backward.hip", "backward_mfma.hip", "rope.hip"]
ARCH = "gfx950"

HIPCC_FLAGS = [
    "--offload-arch=" + ARCH, "-O3", "-std=c++17", "-fPIC",
    # no packed-fp32 instructions in device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # MFMA accumulators in ordinary VGPRs (no AGPR round trips next to the
    # softmax VALU work)
    "-mllvm", "-amdgpu-mfma-vgpr-form",
    # no NaN inputs are produced or expected (masked scores are -inf): run with
    # IEEE mode off so min/max need no quieting of their operands
    "-mno-amdgpu-ieee", "-fno-honor-nans",
    "-I", os.path.join(ROOT, "include"),
]


def _hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    return "hipcc"


def build(verbose: bool = False) -> str:
    """Compile every source and link libdar.so (always recompiles)."""
    build_dir = os.path.join(PKG, "_build")
    os.makedirs(build_dir, exist_ok=True)
    objs = []
    procs = []
    for src in SOURCES:
        obj = os.path.join(build_dir, src.replace(".hip", ".o"))
        cmd = [_hipcc(), *HIPCC_FLAGS, "-c", os.path.join(CSRC, src), "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        procs.append((subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT), src))
        objs.append(obj)
    failed = []
    for p, src in procs:
        out, _ = p.communicate()
        text = out.decode(errors="replace")
        # hipcc's host pass does not know the packed-fp32 feature; that note is harmless
        lines = [l for l in text.splitlines() if "packed-fp32-ops" not in l]
        if lines and (verbose or p.returncode != 0):
            print("\n".join(lines), file=sys.stderr)
        if p.returncode != 0:
            failed.append(src)
    if failed:
        raise RuntimeError("hipcc failed for: " + ", ".join(failed))
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [_hipcc(), "--offload-arch=" + ARCH, "-shared", "-fPIC", *objs, "-o", tmp]
    subprocess.check_call(cmd)
    os.replace(tmp, LIB)
    build_k0(verbose)
    return LIB


def build_k0(verbose: bool = False) -> str:
    """The machine microbenchmarks (include/dar_k0.h) as their own library:
    they are measurement code, not part of the attention path."""
    tmp = K0_LIB + ".tmp%d" % os.getpid()
    cmd = [_hipcc(), *HIPCC_FLAGS, "-shared", os.path.join(CSRC, K0_SOURCE), "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    p = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT)
    text = "\n".join(l for l in p.stdout.decode(errors="replace").splitlines()
                     if "packed-fp32-ops" not in l)
    if p.returncode != 0:
        print(text, file=sys.stderr)
        raise RuntimeError("hipcc failed for " + K0_SOURCE)
    os.replace(tmp, K0_LIB)
    return K0_LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
