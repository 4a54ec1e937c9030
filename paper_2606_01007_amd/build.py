"""Build libtacg.so (the HIP kernels and the C ABI) for gfx950 with hipcc, in-tree.

    python -m paper_2606_01007_amd.build

Every HIP translation unit under csrc/ is compiled to an object in _build/ (in parallel) and linked
into paper_2606_01007_amd/libtacg.so.  Packed-FP32 instruction selection is disabled for all device
code.

build(sanitize=True, out=path) makes a second library whose host code (argument checks, workspace
sizing, launch set-up) carries AddressSanitizer and UndefinedBehaviorSanitizer; device code is built
as usual.  It is loaded with TACG_LIBRARY=path and the clang ASan runtime preloaded (host_asan_runtime()).
"""
from __future__ import annotations

import concurrent.futures as cf
import glob
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libtacg.so")
ARCH = os.environ.get("TACG_OFFLOAD_ARCH", "gfx950")

HIPCC = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-result",
    f"-I{INCLUDE}", f"-I{CSRC}",
]


# host-only sanitizer flags: every -fsanitize is behind -Xarch_host, device code stays uninstrumented
SANITIZE_HOST = ["-Xarch_host", "-g", "-Xarch_host", "-fno-omit-frame-pointer",
                 "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                 "-Xarch_host", "-fno-sanitize-recover=undefined"]


def host_asan_runtime() -> str:
    """Path of the clang ASan runtime that a host-sanitized libtacg.so needs preloaded."""
    clang = os.path.join(os.path.dirname(os.path.realpath(HIPCC)), "..", "llvm", "bin", "clang")
    if not os.path.exists(clang):
        clang = "/opt/rocm/llvm/bin/clang"
    r = subprocess.run([clang, "-print-file-name=libclang_rt.asan-x86_64.so"], capture_output=True, text=True,
                       check=True)
    return r.stdout.strip()


def _compile(src: str, build_dir: str = BUILD, sanitize: bool = False) -> str:
    obj = os.path.join(build_dir, os.path.basename(src) + ".o")
    flags = [f if f != "-O3" else "-O1" for f in FLAGS] + SANITIZE_HOST if sanitize else FLAGS
    cmd = [HIPCC, *flags, "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stdout}\n{r.stderr}")
    return obj


def build(verbose: bool = False, sanitize: bool = False, out: str | None = None) -> str:
    """Compile every csrc/*.hip and link libtacg.so (or `out`).  Always recompiles."""
    lib = out or LIB
    build_dir = os.path.join(BUILD, "sanitize") if sanitize else BUILD
    os.makedirs(build_dir, exist_ok=True)
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")))
    with cf.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        objs = list(ex.map(lambda s: _compile(s, build_dir, sanitize), srcs))
    tmp = lib + ".tmp%d" % os.getpid()
    extra = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined", "-shared-libsan"] \
        if sanitize else []
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *extra, *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, lib)
    if verbose:
        print(f"built {lib}")
    return lib


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
