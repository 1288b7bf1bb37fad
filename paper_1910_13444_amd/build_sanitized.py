"""Build a host-sanitized copy of libpigan.so for the CPU tests of the
argument checks: the C-ABI layer (pigan_api.cpp: descriptor checks,
workspace planning, dispatch) is compiled with AddressSanitizer and
UndefinedBehaviorSanitizer on its host code; the kernel sources are linked
from the ordinary build's objects (built here when missing).

    python -m paper_1910_13444_amd.build_sanitized

The library lands in _build/san/libpigan_san.so.  Load it through
PIGAN_LIBRARY with the sanitizer runtime preloaded (ASAN_RUNTIME below).
"""
from __future__ import annotations

import concurrent.futures as cf
import glob
import os
import subprocess

from . import build as _plain
from .build import BUILD, CSRC, SOURCES, common_flags, hipcc

SAN = os.path.join(BUILD, "san")
LIB_SAN = os.path.join(SAN, "libpigan_san.so")
# each sanitizer flag applies to the host compilation only
HOST_SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer", "-g"]


def asan_runtime() -> str:
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    hits = sorted(glob.glob(os.path.join(rocm, "llvm", "lib", "clang", "*", "lib", "linux",
                                         "libclang_rt.asan-x86_64.so")))
    if not hits:
        raise RuntimeError("the clang AddressSanitizer runtime is not installed")
    return hits[-1]


def _compile(src: str) -> str:
    obj = os.path.join(SAN, src + ".o")
    cmd = [hipcc(), *common_flags(), *HOST_SAN, "-c", os.path.join(CSRC, src), "-o", obj]
    if src.endswith(".cpp"):
        cmd.insert(1, "-xhip")
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stdout}\n{r.stderr}")
    return obj


SANITIZED = ("pigan_api.cpp",)


def _object(src: str) -> str:
    if src in SANITIZED:
        return _compile(src)
    obj = os.path.join(BUILD, src + ".o")
    if not os.path.exists(obj) or os.path.getmtime(obj) < os.path.getmtime(os.path.join(CSRC, src)):
        os.makedirs(BUILD, exist_ok=True)
        obj = _plain._compile(src)
    return obj


def build_sanitized(jobs: int = 4) -> str:
    os.makedirs(SAN, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=max(1, jobs)) as ex:
        objs = list(ex.map(_object, SOURCES))
    cmd = [hipcc(), "--offload-arch=gfx950", "-shared", "-fPIC", "-shared-libsan", *HOST_SAN, *objs,
           "-o", LIB_SAN]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}\n{r.stderr}")
    return LIB_SAN


if __name__ == "__main__":
    print(build_sanitized(min(8, os.cpu_count() or 4)))
