"""Build libsteel.so in-tree with hipcc for gfx950.

    python -m paper_2607_09385_amd.build

Each source compiles to its own object under ``_build/`` (in parallel), then
one link produces ``paper_2607_09385_amd/libsteel.so``.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libsteel.so")
SOURCES = ["steel_api.cpp", "block_index.hip", "block_select.hip", "attn_fwd.hip", "attn_ws.hip",
           "quant_fp8.hip",
           "attn_merge.hip", "noalloc.hip", "mfma_peak.hip"]
ARCH = "gfx950"

# Packed fp32 VALU forms are kept out of every code object: the compiler would
# otherwise fuse pairs of scalar float ops into them.
COMMON = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wno-unused-command-line-argument",
]
# Both attention sources keep the compiler's MFMA accumulators in VGPRs: the
# softmax reads the scores with VALU instructions (AGPR-resident scores would
# cost a copy per element), and attn_ws.hip runs two waves per SIMD, whose
# 256 registers each hold no AGPR file.
PER_SOURCE = {"attn_fwd.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form=1"],
              "attn_ws.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form=1"]}


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found: libsteel needs ROCm's hipcc to build")


def _compile(src: str, extra: list[str]) -> str:
    obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
    lang = ["-x", "hip"] if src.endswith(".hip") else []
    cmd = [hipcc(), *COMMON, *PER_SOURCE.get(src, []), *extra, *lang, "-c", os.path.join(CSRC, src),
           "-o", obj]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"compiling {src} failed:\n{' '.join(cmd)}\n{res.stdout}\n{res.stderr}")
    return obj


def build(extra: list[str] | None = None, verbose: bool = False) -> str:
    """Compile every source and link libsteel.so; returns its path."""
    extra = list(extra or [])
    os.makedirs(BUILD, exist_ok=True)
    with ThreadPoolExecutor(max_workers=len(SOURCES)) as ex:
        objs = list(ex.map(lambda s: _compile(s, extra), SOURCES))
    tmp = LIB + ".tmp"
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"linking libsteel.so failed:\n{' '.join(cmd)}\n{res.stdout}\n{res.stderr}")
    os.replace(tmp, LIB)
    if verbose:
        print(f"built {LIB}")
    return LIB


if __name__ == "__main__":
    build(sys.argv[1:], verbose=True)
