"""Build libsoap.so (HIP, gfx950) and the input generator in-tree."""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libsoap.so")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

HIP_FLAGS = [
    "-O3", "-fPIC", "-std=c++17", f"--offload-arch={ARCH}",
    # keep the compiler from emitting packed fp32 arithmetic
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # matrix-core accumulators in ordinary VGPRs: the accumulation chains are
    # loop-carried, and the AGPR form copies them out and back per MFMA
    "-mllvm", "-amdgpu-mfma-vgpr-form",
    "-I", os.path.join(ROOT, "include"), "-I", CSRC,
]
HOST_FLAGS = ["-O2", "-fPIC", "-std=gnu++17", "-fext-numeric-literals", "-I", os.path.join(ROOT, "include"), "-I", CSRC]

HIP_SOURCES = ["neighbors.hip", "soap_kernels.hip", "density_streamed.hip"]
HIP_HOST_SOURCES = ["api.cpp"]
HOST_SOURCES = ["basis.cpp"]


def _run(cmd):
    print(" ".join(cmd), flush=True)
    subprocess.check_call(cmd)


# the float32 Jacobian kernel for fixed basis sizes, in parts built in parallel
FIXED_SOURCE, FIXED_PARTS = "jacobian_fixed.hip", 3


def build(verbose: bool = True) -> str:
    from concurrent.futures import ThreadPoolExecutor
    os.makedirs(BUILD, exist_ok=True)
    jobs = []
    for src in HIP_SOURCES + HIP_HOST_SOURCES:
        obj = os.path.join(BUILD, src + ".o")
        lang = [] if src.endswith(".hip") else ["-x", "hip"]
        jobs.append((obj, [HIPCC, *HIP_FLAGS, *lang, "-c", os.path.join(CSRC, src), "-o", obj]))
    for part in range(FIXED_PARTS):
        obj = os.path.join(BUILD, f"{FIXED_SOURCE}.{part}.o")
        jobs.append((obj, [HIPCC, *HIP_FLAGS, f"-DJF_PART={part}", "-c", os.path.join(CSRC, FIXED_SOURCE), "-o", obj]))
    with ThreadPoolExecutor(max_workers=min(len(jobs), os.cpu_count() or 1)) as ex:
        list(ex.map(lambda j: _run(j[1]), jobs))
    objs = [j[0] for j in jobs]
    for src in HOST_SOURCES:
        obj = os.path.join(BUILD, src + ".o")
        _run(["g++", *HOST_FLAGS, "-c", os.path.join(CSRC, src), "-o", obj])
        objs.append(obj)
    tmp = LIB + ".tmp%d" % os.getpid()
    _run([HIPCC, "-shared", f"--offload-arch={ARCH}", "-o", tmp, *objs, "-lquadmath"])
    os.replace(tmp, LIB)
    from . import workloads
    workloads.build_generator(force=True)
    return LIB


if __name__ == "__main__":
    build()
    sys.exit(0)
