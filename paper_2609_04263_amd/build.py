"""Build libkvq.so (the HIP kernels and the C ABI of include/kvq.h) for gfx950.

Every source is compiled by hipcc for gfx950 only, in-tree, into
``paper_2609_04263_amd/libkvq.so``.  Flags that matter for results:

* ``-fhip-fp32-correctly-rounded-divide-sqrt`` and
  ``-fno-gpu-flush-denormals-to-zero``: IEEE binary32 division and denormals,
  so the coder's scales and codes are bit-exact;
* ``-ffp-contract=off`` for ``append.hip`` (no fused multiply-add in the coder);
* packed fp32 instructions disabled for all device code;
* mixed-precision FMA instructions (v_fma_mix*/v_mad_mix*) disabled: the
  attention kernel splits fp32 operands into fp16 hi + lo parts, and on
  gfx950 the fused fp16(a*b - c) these instructions provide was measured to
  deviate from the fp32 fused result by up to ~1e-4 relative, which the
  split must not lose.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libkvq.so")
ROOT = os.path.dirname(HERE)

SOURCES = ["kvq_api.cpp", "append.hip", "attn.hip", "attn_d64.hip", "attn_d128.hip", "attn_d256.hip",
           "project.hip", "merge.hip", "prefill.hip"]
# MFMA accumulators in VGPRs: the attention loop rescales them with VALU
# instructions, and AGPR accumulators cost a copy each way per block.
_VGPR_MFMA = ["-mllvm", "-amdgpu-mfma-vgpr-form"]
PER_FILE = {"append.hip": ["-ffp-contract=off"], "attn_d64.hip": _VGPR_MFMA, "attn_d128.hip": _VGPR_MFMA,
            "attn_d256.hip": _VGPR_MFMA}


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found: the HIP library cannot be built")


def common_flags() -> list[str]:
    return ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-Wall",
            "-fhip-fp32-correctly-rounded-divide-sqrt", "-fno-gpu-flush-denormals-to-zero",
            "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
            "-Xclang", "-target-feature", "-Xclang", "-fma-mix-insts",
            "-I", os.path.join(ROOT, "include")]


def _compile(src: str) -> str:
    obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
    cmd = [hipcc(), *common_flags(), *PER_FILE.get(src, []), "-x", "hip", "-c",
           os.path.join(CSRC, src), "-o", obj]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{res.stdout}\n{res.stderr}")
    return obj


def build(verbose: bool = False) -> str:
    """Compile every source and link libkvq.so; returns its path."""
    os.makedirs(BUILD, exist_ok=True)
    with ThreadPoolExecutor(max_workers=len(SOURCES)) as ex:
        objs = list(ex.map(_compile, SOURCES))
    tmp = LIB + ".tmp"
    cmd = [hipcc(), "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", tmp]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"link failed:\n{res.stdout}\n{res.stderr}")
    os.replace(tmp, LIB)
    if verbose:
        print(f"built {LIB}")
    return LIB


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
