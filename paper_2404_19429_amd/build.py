"""Build liblancet_moe.so in-tree with hipcc for gfx950.

Usage: python -m paper_2404_19429_amd.build [-v]
Every source is compiled to an object under _build/ (in parallel), then
linked into paper_2404_19429_amd/liblancet_moe.so.  Always recompiles.
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
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "liblancet_moe.so")
SOURCES = ["api.cpp", "block.cpp", "plan.cpp", "gate.hip", "route.hip", "gemm.hip", "attn.hip", "norm.hip"]
ARCH = "gfx950"

HIPCC_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wno-unused-result", "-I", INCLUDE, "-I", CSRC,
]


def _hipcc() -> str:
    h = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(h):
        raise RuntimeError("hipcc not found; ROCm is required to build the HIP library")
    return h


def _compile(src: str, verbose: bool) -> str:
    obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
    cmd = [_hipcc(), "-x", "hip", "-c", os.path.join(CSRC, src), "-o", obj] + HIPCC_FLAGS
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    msgs = [ln for ln in (r.stdout + r.stderr).splitlines() if "packed-fp32-ops" not in ln]
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n" + "\n".join(msgs))
    if verbose and msgs:
        print("\n".join(msgs), flush=True)
    return obj


ASM_READ_SOURCES = ["gemm.hip", "attn.hip"]  # kernels that read LDS through inline asm


def _check_isa(src: str, verbose: bool) -> None:
    """Refuse a build whose kernels use an inline-asm LDS read before its wait."""
    from paper_2404_19429_amd.isa_check import check_text
    out = os.path.join(BUILD, os.path.splitext(src)[0] + ".s")
    cmd = [_hipcc(), "-x", "hip", "-S", "--offload-device-only", os.path.join(CSRC, src), "-o", out] + HIPCC_FLAGS
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc -S failed on {src}:\n" + r.stderr)
    bad = check_text(open(out).read(), "_ZN4lmoe")
    if bad:
        detail = "\n".join(f"{k}: {v[:3]}" for k, v in bad.items())
        raise RuntimeError(f"ISA check failed on {src}: asm LDS read results used before their wait\n" + detail)
    if verbose:
        print(f"ISA check passed: {src}", flush=True)


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=min(8, len(SOURCES) + len(ASM_READ_SOURCES))) as ex:
        isa = [ex.submit(_check_isa, s, verbose) for s in ASM_READ_SOURCES]
        objs = list(ex.map(lambda s: _compile(s, verbose), SOURCES))
        for f in isa:
            f.result()
    tmp = LIB + ".tmp"
    cmd = [_hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp] + objs
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n" + r.stdout + r.stderr)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    if ROOT not in sys.path:
        sys.path.insert(0, ROOT)
    print(build(verbose="-v" in sys.argv))
