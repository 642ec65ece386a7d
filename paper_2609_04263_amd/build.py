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

# MFMA accumulators in VGPRs: the attention loop rescales them with VALU
# instructions, and AGPR accumulators cost a copy each way per block.
_VGPR_MFMA = ["-mllvm", "-amdgpu-mfma-vgpr-form"]
# (source, object name, extra flags).  The decode split kernels are built
# from one source, once per (head size, metadata width, key axis) family.
UNITS = [("kvq_api.cpp", "kvq_api", []), ("append.hip", "append", ["-ffp-contract=off"]),
         ("attn.hip", "attn", _VGPR_MFMA), ("project.hip", "project", []), ("merge.hip", "merge", []),
         ("prefill.hip", "prefill", [])]
UNITS += [("attn_part.hip", f"attn_{d}_{m}_{pc}",
           _VGPR_MFMA + [f"-DKVQ_PART_D={d}", f"-DKVQ_PART_M16={m}", f"-DKVQ_PART_PC={pc}"])
          for d in (64, 128, 256) for m in (0, 1) for pc in (0, 1)]
SOURCES = sorted({u[0] for u in UNITS})


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


def _compile(unit) -> str:
    src, name, extra = unit
    obj = os.path.join(BUILD, name + ".o")
    cmd = [hipcc(), *common_flags(), *extra, "-x", "hip", "-c", os.path.join(CSRC, src), "-o", obj]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed for {name} ({src}):\n{res.stdout}\n{res.stderr}")
    return obj


def build(verbose: bool = False, units=None) -> str:
    """Compile every unit (or the named objects) and link libkvq.so; returns its path."""
    os.makedirs(BUILD, exist_ok=True)
    todo = UNITS if units is None else [u for u in UNITS if u[1] in units]
    workers = max(1, min(len(todo), os.cpu_count() or 1))
    with ThreadPoolExecutor(max_workers=workers) as ex:
        list(ex.map(_compile, todo))
    objs = [os.path.join(BUILD, u[1] + ".o") for u in UNITS]
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
