"""Build libhma.so (gfx950) in-tree with hipcc.

    python -m paper_2606_29986_amd.build

The library is compiled for gfx950 only, with packed-FP32 instruction
selection disabled (plain float code must not be turned into v_pk_* FP32
ops).  FP32 denormals stay enabled (the HIP default): BF16 subnormals are
produced through FP32 denormals in the BFP8 decode.
"""
from __future__ import annotations

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libhma.so")

SOURCES = ["hma_api.cpp", "bfp8_dequant.hip", "decode_attn.hip", "rebuild_tiled.hip", "read_probe.hip",
           "valu_attn.hip"]
ARCH = "gfx950"


def hipcc_command(out: str, extra=()) -> list:
    cmd = ["hipcc", f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-shared",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-fvisibility=hidden", "-Wall", "-Wno-unused-command-line-argument", "-Wno-inline-asm",
           f"-I{INCLUDE}", f"-I{CSRC}", *extra, "-x", "hip"]
    cmd += [os.path.join(CSRC, s) for s in SOURCES]
    cmd += ["-o", out]
    return cmd


def build(verbose: bool = False, extra=()) -> str:
    """Compile every HIP source into paper_2606_29986_amd/libhma.so (always)."""
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = hipcc_command(tmp, extra)
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    # hipcc's host pass does not know the packed-fp32 feature; that warning is expected
    noise = "'-packed-fp32-ops' is not a recognized feature"
    err = "\n".join(l for l in res.stderr.splitlines() if noise not in l)
    if res.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + err)
    if verbose and err.strip():
        print(err, file=sys.stderr)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
