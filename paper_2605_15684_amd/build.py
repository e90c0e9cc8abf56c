"""Build libssba.so (HIP kernels + C ABI) for gfx950 with hipcc, in-tree.

    python -m paper_2605_15684_amd.build          # compile and link
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
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libssba.so")
ARCH = os.environ.get("SSBA_OFFLOAD_ARCH", "gfx950")

SOURCES = {
    "ssba_api.cpp": [],
    "ssba_select.cpp": [],
    # fp64 gate: no contraction of multiply-add, so lists are bit-reproducible.
    "ssba_index.hip": ["-ffp-contract=off"],
    "ssba_attn_bf16.hip": [],
    "ssba_attn_f32.hip": [],
    # MFMA results in ordinary VGPRs: the softmax reads every score and the
    # default accumulation-register form costs a copy per element.
    "ssba_attn_mfma.hip": ["-ffp-contract=off", "-mllvm", "-amdgpu-mfma-vgpr-form"],
    "ssba_haar.hip": ["-ffp-contract=off"],
    "ssba_bwd.hip": [],
    "ssba_probe.hip": [],
    "ssba_noalloc.hip": [],
}

COMMON = [
    "-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
    # Packed fp32 VALU forms are switched off for every kernel.
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
    "-I", INCLUDE, "-I", CSRC,
]


def _hipcc() -> str:
    cand = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(cand):
        raise RuntimeError("hipcc not found: the SSBA library needs ROCm's hipcc to build")
    return cand


def _compile(src: str, extra, verbose: bool) -> str:
    obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
    lang = ["-x", "hip"] if src.endswith(".cpp") else []
    cmd = [_hipcc(), *COMMON, *extra, *lang, "-c", os.path.join(CSRC, src), "-o", obj]
    res = subprocess.run(cmd, capture_output=True, text=True)
    noise = "is not a recognized feature for this target"
    err = "\n".join(l for l in (res.stderr or "").splitlines() if noise not in l)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{' '.join(cmd)}\n{err}")
    if verbose and err.strip():
        print(err, file=sys.stderr)
    return obj


def build(verbose: bool = False) -> str:
    """Compile every kernel source and link ``libssba.so``; returns its path."""
    os.makedirs(BUILD, exist_ok=True)
    with ThreadPoolExecutor(max_workers=min(4, os.cpu_count() or 1)) as ex:
        objs = list(ex.map(lambda kv: _compile(kv[0], kv[1], verbose), SOURCES.items()))
    tmp = LIB + ".tmp"
    cmd = [_hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"link failed:\n{' '.join(cmd)}\n{res.stderr}")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
