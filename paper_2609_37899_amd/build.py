"""Build ``libsoma.so`` (the HIP library behind include/soma.h) for gfx950.

Run ``python -m paper_2609_37899_amd.build`` (or ``__graft_entry__.build()``).
The library is built in-tree next to this file.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
SRC = os.path.join(PKG, "csrc", "soma_api.hip")
DEPS = [os.path.join(PKG, "csrc", f) for f in ("soma_api.hip", "soma_kernels.hpp", "soma_body.hpp", "soma_rng.hpp")] + \
       [os.path.join(ROOT, "include", "soma.h")]
LIB = os.path.join(PKG, "libsoma.so")
ARCH = os.environ.get("SOMA_OFFLOAD_ARCH", "gfx950")

HIPCC_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-shared",
    # The probe generator is specified operation by operation: no contraction.
    "-ffp-contract=off",
    # Packed fp32 VALU instructions (v_pk_*_f32) stay off: plain fp32 code
    # is compiled to single-lane instructions only.
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # The instruction scheduler's ILP strategy: the body kernel runs one wave
    # per SIMD, so its latencies are hidden only by independent instructions
    # of the same wave (measured: 35.4 -> 27.2 ms per step on the body
    # workload, 113.4 -> 111.7 ms on the stacked-LSTM workload).
    "-mllvm", "-amdgpu-sched-strategy=max-ilp",
    "-Wall", "-Wno-unused-command-line-argument",
]


def hipcc() -> str:
    return shutil.which("hipcc") or "/opt/rocm/bin/hipcc"


def build(verbose: bool = False) -> str:
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [hipcc(), *HIPCC_FLAGS, "-I", os.path.join(ROOT, "include"), "-I", os.path.join(PKG, "csrc"),
           "-o", tmp, SRC]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.check_call(cmd, cwd="/tmp")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
