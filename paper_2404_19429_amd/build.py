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


# Host sources checked under AddressSanitizer and UndefinedBehaviorSanitizer
# (the C-ABI validation, the planners and the block's host orchestration).
# Their device-free objects are rebuilt with the sanitizers on the host side
# only and linked with the regular objects of the kernel sources.
SANITIZED_SOURCES = ["api.cpp", "plan.cpp", "block.cpp"]
SANITIZE_HOST = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                 "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host", "-fno-omit-frame-pointer"]


def asan_runtime() -> str:
    """The compiler's AddressSanitizer runtime (to preload into a host process that loads the sanitized library)."""
    clang = os.path.join(os.path.dirname(os.path.realpath(_hipcc())), "..", "llvm", "bin", "clang")
    if not os.path.exists(clang):
        clang = "/opt/rocm/llvm/bin/clang"
    r = subprocess.run([clang, "--print-file-name=libclang_rt.asan-x86_64.so"], capture_output=True, text=True)
    return r.stdout.strip()


def build_host_sanitized(verbose: bool = False) -> str:
    """_build/san/liblancet_moe_san.so: SANITIZED_SOURCES with host-side ASan/UBSan,
    the kernel sources' objects from the last regular build (which must exist)."""
    san = os.path.join(BUILD, "san")
    os.makedirs(san, exist_ok=True)
    others = [os.path.join(BUILD, os.path.splitext(s)[0] + ".o") for s in SOURCES if s not in SANITIZED_SOURCES]
    missing = [o for o in others if not os.path.exists(o)]
    if missing:
        raise FileNotFoundError("run the regular build first; missing " + ", ".join(missing))

    def one(src):
        obj = os.path.join(san, os.path.splitext(src)[0] + ".o")
        flags = [f for f in HIPCC_FLAGS if f != "-O3"] + ["-O1", "-g"] + SANITIZE_HOST
        cmd = [_hipcc(), "-x", "hip", "-c", os.path.join(CSRC, src), "-o", obj] + flags
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"hipcc (sanitized) failed on {src}:\n{r.stderr}")
        return obj

    with cf.ThreadPoolExecutor(max_workers=len(SANITIZED_SOURCES)) as ex:
        objs = list(ex.map(one, SANITIZED_SOURCES))
    lib = os.path.join(san, "liblancet_moe_san.so")
    cmd = ([_hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", lib] + objs + others +
           ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined", "-Xarch_host", "-shared-libsan"])
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("sanitized link failed:\n" + r.stdout + r.stderr)
    return lib


if __name__ == "__main__":
    if ROOT not in sys.path:
        sys.path.insert(0, ROOT)
    print(build(verbose="-v" in sys.argv))
