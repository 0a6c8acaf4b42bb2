"""Build libbla.so (the HIP library behind include/bla.h) for gfx950 with hipcc.

Every translation unit under csrc/ is compiled in parallel into _build/ at the
repository root, then linked into paper_2606_09862_amd/libbla.so.  Run as
``python -m paper_2606_09862_amd.build`` or through ``__graft_entry__.build()``.
"""
from __future__ import annotations

import concurrent.futures as cf
import glob
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libbla.so")

ARCH = "gfx950"
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
# Packed fp32 instructions are disabled for every HIP translation unit.  Matrix-core
# accumulators are allocated in ordinary VGPRs (the kernels post-process every
# accumulator with vector ALU code, which cannot read AGPRs directly).
CFLAGS = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}", f"-I{INCLUDE}", f"-I{CSRC}",
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", "-Wno-unused-result",
          "-mllvm", "-amdgpu-mfma-vgpr-form"]


# Units whose kernels the compiler cannot build with VGPR-form accumulators (or that need the
# accumulation registers as well: the backward kernels hold four state tiles per wave).
NO_VGPR_FORM = {"bla_fwd_bf16_d128_wide.hip", "bla_fwd_f32_d128.hip", "bla_bwd_bf16.hip", "bla_bwd_f32.hip"}


def _compile(src: str) -> str:
    obj = os.path.join(BUILD, os.path.basename(src) + ".o")
    flags = list(CFLAGS)
    if os.path.basename(src) in NO_VGPR_FORM:
        flags = flags[:-2]
    cmd = [HIPCC, *flags, "-c", src, "-o", obj]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{res.stdout}\n{res.stderr}")
    return obj


def build(jobs: int | None = None) -> str:
    os.makedirs(BUILD, exist_ok=True)
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")))
    jobs = jobs or min(len(srcs), os.cpu_count() or 4, 16)
    with cf.ThreadPoolExecutor(max_workers=jobs) as ex:
        objs = list(ex.map(_compile, srcs))
    tmp = LIB + ".tmp"
    cmd = [HIPCC, "-shared", "-fPIC", f"--offload-arch={ARCH}", *objs, "-o", tmp, "-lhipblaslt"]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"link failed:\n{res.stdout}\n{res.stderr}")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(int(sys.argv[1]) if len(sys.argv) > 1 else None))
