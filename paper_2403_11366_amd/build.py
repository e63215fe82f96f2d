"""Build the gfx950 HIP library liblora_linear.so in-tree with hipcc.

Usage: python -m paper_2403_11366_amd.build   (or call build()).
Objects go to paper_2403_11366_amd/_build/; the shared library is written next
to this file, where the Python binding loads it from.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "liblora_linear.so")
SOURCES = ["lora_abi.cpp", "lora_fwd.hip", "lora_bwd.hip", "lora_merge.hip", "lora_mask.hip"]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (set HIPCC or install ROCm under /opt/rocm)")


FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-result", "-Wno-unused-function",
]


def _compile(src: str) -> str:
    obj = os.path.join(BUILD, os.path.basename(src) + ".o")
    # HIP sources keep their intermediate files (-save-temps=obj): the device
    # object is assembled from the saved gfx950 assembly, which asm_check reads.
    lang = ["-x", "hip", "-save-temps=obj"] if src.endswith(".hip") else []
    cmd = [hipcc()] + FLAGS + ["-I", os.path.join(ROOT, "include"), "-I", CSRC] + lang + \
          ["-c", os.path.join(CSRC, src), "-o", obj]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n{res.stderr}")
    return obj


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=len(SOURCES)) as ex:
        objs = list(ex.map(_compile, SOURCES))
    # kernels whose LDS reads are inline assembly: no register of a read may be
    # touched before its wait, no scratch, no calls (asm_check)
    from paper_2403_11366_amd import asm_check
    device_asm = [os.path.join(BUILD, os.path.splitext(s)[0] + "-hip-amdgcn-amd-amdhsa-gfx950.s")
                  for s in SOURCES if s.endswith(".hip")]
    problems = asm_check.check_files(device_asm)
    if problems:
        raise RuntimeError("inline-assembly LDS reads unsafe in the compiled kernels:\n" + "\n".join(problems[:20]))
    if verbose:
        print(f"asm_check: {asm_check.count_checked(device_asm)} kernel(s) with inline-asm LDS reads verified")
    tmp = LIB + ".tmp"
    cmd = [hipcc(), "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp] + objs
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"link failed:\n{res.stderr}")
    os.replace(tmp, LIB)
    if verbose:
        print(f"built {LIB}")
    return LIB


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
