"""Build librrs.so (the C-ABI HIP library) in-tree for gfx950 with hipcc.

Each source is compiled to an object in parallel, then linked into
paper_2409_20361_amd/librrs.so. Always recompiles.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "librrs.so")
OBJDIR = os.path.join(PKG, "_build")

SOURCES = ["rrs_api.cpp", "rrs_quant.hip", "rrs_weight.hip", "rrs_gemm.hip", "rrs_gemm_small.hip",
           "rrs_gemm_decode.hip", "rrs_quant_wave.hip", "rrs_reorder.hip", "rrs_quant_rows.hip",
           "rrs_gemm_stream.hip", "rrs_gemm_stream_gather.hip", "rrs_noalloc.hip"]

# Per-source code-generation options on top of COMMON.
# rrs_gemm_stream_gather.hip: keep MFMA results in VGPRs (the per-block
#   rescale reads every accumulator; in AGPRs each read is an extra copy).
EXTRA = {"rrs_gemm_stream_gather.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"]}

# -packed-fp32-ops: no v_pk_{add,mul,fma}_f32 in any kernel.
# -ffp-contract=off: every rounding in the rotation and scale chain is an
#   explicit single IEEE operation; the GEMM epilogue asks for fma explicitly.
COMMON = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-ffp-contract=off", "-fno-fast-math",
    "-Wall", "-Wno-unused-function", "-Wno-unknown-warning-option",
    "-I" + INCLUDE, "-I" + CSRC,
]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build librrs.so)")


def _compile(src: str) -> str:
    obj = os.path.join(OBJDIR, os.path.splitext(src)[0] + ".o")
    lang = ["-x", "hip"] if src.endswith(".hip") else []
    cmd = [hipcc()] + COMMON + EXTRA.get(src, []) + ["-c"] + lang + [os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    # hipcc's host pass does not know the packed-fp32 feature; that warning is expected.
    noise = [ln for ln in r.stderr.splitlines()
             if ln.strip() and "packed-fp32-ops" not in ln and "not a recognized feature" not in ln]
    if noise:
        sys.stderr.write(f"[build] {src}:\n" + "\n".join(noise) + "\n")
    return obj


def build(verbose: bool = False) -> str:
    os.makedirs(OBJDIR, exist_ok=True)
    with ThreadPoolExecutor(max_workers=min(len(SOURCES), os.cpu_count() or 4)) as ex:
        objs = list(ex.map(_compile, SOURCES))
    tmp = LIB + ".tmp"
    cmd = [hipcc(), "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp] + objs
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, LIB)
    if verbose:
        print(f"[build] wrote {LIB}")
    return LIB


if __name__ == "__main__":
    build(verbose=True)
