"""Build libppd.so (HIP kernels + C ABI host code) for gfx950 with hipcc.

    python -m paper_2405_18628_amd.build          # or build() from Python

Objects go to paper_2405_18628_amd/_build/, the library next to this file.
Every call rebuilds (the sources are small; a full build takes well under a
minute on 8 cores).
"""
from __future__ import annotations

import concurrent.futures as cf
import glob
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
OUT = os.path.join(HERE, "libppd.so")
BUILD = os.path.join(HERE, "_build")
ARCH = os.environ.get("PPD_OFFLOAD_ARCH", "gfx950")

HIPCC = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
# packed-fp32 instructions are disabled for all device code: some of their
# forms have produced silently wrong results on this hardware
FLAGS = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-Wno-unused-command-line-argument"]


def _compile(src: str) -> str:
    obj = os.path.join(BUILD, os.path.basename(src) + ".o")
    cmd = [HIPCC, *FLAGS, "-x", "hip", "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stderr}")
    return obj


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")) + glob.glob(os.path.join(CSRC, "*.cpp")))
    with cf.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        objs = list(ex.map(_compile, srcs))
    tmp = OUT + ".tmp"
    cmd = [HIPCC, *FLAGS, "-shared", "-o", tmp, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stderr}")
    os.replace(tmp, OUT)
    if verbose:
        print(f"built {OUT}")
    return OUT


# host sanitizers: every -fsanitize applies to the host compilation only
HOST_SANITIZE = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                 "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer"]
SANITIZED = os.path.join(BUILD, "libppd_hostsan.so")


def build_host_sanitized(verbose: bool = False) -> str:
    """_build/libppd_hostsan.so: the host sources (argument checks, tree
    builders, workspace layout, launch sequencing) compiled with
    AddressSanitizer and UndefinedBehaviorSanitizer and linked with the device
    objects of the last build().  Load it with the sanitizer runtime
    preloaded (sanitizer_runtime()) and PPD_LIBRARY pointing at it."""
    hosts = sorted(glob.glob(os.path.join(CSRC, "*.cpp")))
    devs = [os.path.join(BUILD, os.path.basename(f) + ".o")
            for f in sorted(glob.glob(os.path.join(CSRC, "*.hip")))]
    if not all(os.path.exists(o) for o in devs):
        build()
    objs = []
    for src in hosts:
        obj = os.path.join(BUILD, os.path.basename(src) + ".hostsan.o")
        cmd = [HIPCC, *FLAGS, *HOST_SANITIZE, "-x", "hip", "-c", src, "-o", obj]
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"hipcc (host sanitizers) failed for {src}:\n{r.stderr}")
        objs.append(obj)
    cmd = [HIPCC, *FLAGS, "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-shared-libasan", "-shared", "-o", SANITIZED, *objs, *devs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link (host sanitizers) failed:\n{r.stderr}")
    if verbose:
        print(f"built {SANITIZED}")
    return SANITIZED


def sanitizer_runtime() -> str:
    """The compiler's shared AddressSanitizer runtime (to preload into a
    Python process that loads the sanitized library)."""
    cands = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    if not cands:
        raise RuntimeError("libclang_rt.asan-x86_64.so not found under /opt/rocm/llvm")
    return cands[-1]


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
