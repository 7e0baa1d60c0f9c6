"""Build libfqvit.so (the gfx950 HIP kernels and their C ABI) in the package
directory with hipcc."""
from __future__ import annotations

import concurrent.futures
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libfqvit.so")
SOURCES = ["ptf_layernorm.hip", "lis_attention.hip", "lis_inst_lo.hip", "lis_inst_hi.hip",
           "lis_inst_unit.hip", "ptf_quant.hip", "lis_qk.hip", "lis_qk_dk32.hip",
           "lis_qk_dk64.hip", "lis_long_lo.hip", "lis_long_hi.hip",
           "lis_qk_long.hip", "lis_attn_v.hip",
           "fqvit_abi.cpp"]
OBJDIR = os.path.join(HERE, "_build")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    # IEEE double evaluated exactly as written (the LayerNorm factors must match
    # the definition bit for bit): no contraction into fused multiply-adds.
    "-ffp-contract=off",
    # no packed-FP32 instructions
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
]


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError("hipcc failed: " + " ".join(cmd))


def build(verbose: bool = False) -> str:
    """Compile every translation unit in parallel, then link libfqvit.so."""
    os.makedirs(OBJDIR, exist_ok=True)
    inc = ["-I", os.path.join(ROOT, "include"), "-I", CSRC]
    cflags = [f for f in FLAGS if f != "-shared"]
    objs = [os.path.join(OBJDIR, s + ".o") for s in SOURCES]
    jobs = [[HIPCC, *cflags, *inc, "-c", os.path.join(CSRC, s), "-o", o]
            for s, o in zip(SOURCES, objs)]
    workers = min(len(jobs), max(1, min(8, os.cpu_count() or 1)))
    with concurrent.futures.ThreadPoolExecutor(workers) as ex:
        list(ex.map(lambda c: _run(c, verbose), jobs))
    tmp = LIB + ".tmp"
    _run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", tmp], verbose)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
