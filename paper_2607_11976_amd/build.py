"""Builds the HIP library liblitetopk.so for gfx950, in-tree.

    python -m paper_2607_11976_amd.build

Each translation unit compiles in parallel with hipcc, then they are linked
into one shared object next to this file. Packed FP32 instructions are
disabled (-packed-fp32-ops) for every device compile.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
OUT = os.path.join(HERE, "liblitetopk.so")
OBJDIR = os.path.join(HERE, "_build")
SOURCES = ["abi.hip", "select.hip", "score.hip", "sample.hip", "union.hip", "wide.hip"]
ARCH = os.environ.get("LT_OFFLOAD_ARCH", "gfx950")


def hipcc() -> str:
    for c in (os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "bin", "hipcc"), "hipcc"):
        if os.path.sep not in c or os.path.exists(c):
            return c
    return "hipcc"


def flags() -> list:
    return ["--offload-arch=" + ARCH, "-O3", "-std=c++20", "-fPIC", "-Wall", "-Wno-unused-function",
            "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
            "-I", os.path.join(HERE, "..", "include")]


def _compile(src: str) -> str:
    obj = os.path.join(OBJDIR, os.path.splitext(src)[0] + ".o")
    cmd = [hipcc()] + flags() + ["-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("hipcc failed for %s:\n%s\n%s" % (src, " ".join(cmd), r.stderr))
    return obj


def build(verbose: bool = False) -> str:
    os.makedirs(OBJDIR, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=len(SOURCES)) as ex:
        objs = list(ex.map(_compile, SOURCES))
    tmp = OUT + ".tmp"
    cmd = [hipcc(), "--offload-arch=" + ARCH, "-shared", "-fPIC", "-o", tmp] + objs
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n%s\n%s" % (" ".join(cmd), r.stderr))
    os.replace(tmp, OUT)
    if verbose:
        print("built", OUT)
    return OUT


SAN_OUT = os.path.join(OBJDIR, "liblitetopk_san.so")


def build_sanitized(verbose: bool = False) -> str:
    """The same library with the host code of the C ABI (abi.hip: argument
    checks, workspace sizing and carving) built under AddressSanitizer and
    UndefinedBehaviorSanitizer; the device code and the other translation
    units are the regular objects (built first if missing). The sanitizer
    runtime is not linked in: a process loads it first (LD_PRELOAD of the
    path sanitizer_runtime() returns)."""
    os.makedirs(OBJDIR, exist_ok=True)
    others = [os.path.join(OBJDIR, os.path.splitext(s)[0] + ".o") for s in SOURCES if s != "abi.hip"]
    if not all(os.path.exists(o) for o in others):
        build(verbose=verbose)
    obj = os.path.join(OBJDIR, "abi_san.o")
    cmd = [hipcc()] + flags() + ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                                 "-Xarch_host", "-fno-sanitize-recover=undefined",
                                 "-Xarch_host", "-fno-omit-frame-pointer", "-g",
                                 "-c", os.path.join(CSRC, "abi.hip"), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("hipcc failed for the sanitized abi.hip:\n%s\n%s" % (" ".join(cmd), r.stderr))
    tmp = SAN_OUT + ".tmp"
    cmd = [hipcc(), "--offload-arch=" + ARCH, "-shared", "-fPIC", "-o", tmp, obj] + others
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n%s\n%s" % (" ".join(cmd), r.stderr))
    os.replace(tmp, SAN_OUT)
    if verbose:
        print("built", SAN_OUT)
    return SAN_OUT


def sanitizer_runtime() -> str:
    """Path of the compiler's AddressSanitizer runtime (with the
    UndefinedBehaviorSanitizer handlers), or '' if it is not installed."""
    r = subprocess.run([hipcc(), "-print-file-name=libclang_rt.asan-x86_64.so"], capture_output=True, text=True)
    p = r.stdout.strip()
    if r.returncode == 0 and os.path.isabs(p) and os.path.exists(p):
        return p
    base = os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "llvm", "lib", "clang")
    for v in sorted(os.listdir(base)) if os.path.isdir(base) else []:
        c = os.path.join(base, v, "lib", "linux", "libclang_rt.asan-x86_64.so")
        if os.path.exists(c):
            return c
    return ""


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
