"""Build libagnes.so (HIP, gfx950) in-tree with hipcc.

Every HIP translation unit is compiled with packed FP32 instructions disabled
and linked into one shared library next to this file.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
# AGNES_SANITIZE (e.g. "address,undefined"): the host code is built with
# LLVM's sanitizers (device code unchanged) into a separate library, which
# loads only under the sanitizer runtime (tests/sanitized_cpu_suite.py).
SANITIZE = os.environ.get("AGNES_SANITIZE", "")
LIB = os.path.join(HERE, "libagnes.san.so" if SANITIZE else "libagnes.so")
if SANITIZE:
    BUILD = os.path.join(HERE, "_build_san")
SOURCES = ["prims.hip", "store.hip", "pipeline.hip", "bucket.hip", "sage.hip", "api.hip"]
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
HIPCC = os.environ.get("HIPCC", os.path.join(ROCM, "bin", "hipcc"))
ARCH = "gfx950"
FLAGS = ["--offload-arch=" + ARCH, "-O3", "-std=c++17", "-fPIC", "-Wall",
         "-Wno-unused-function", "-Wno-unused-result",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def _host_sanitizer_flags() -> list:
    """Each sanitizer flag for the host pass only; vptr and function checks
    are left out (they need the C++ parts of the runtime, which a preloaded
    runtime does not bring)."""
    flags = ["-g", "-fno-omit-frame-pointer"]
    for f in ("-fsanitize=" + SANITIZE, "-fno-sanitize=vptr,function", "-fno-sanitize-recover=all"):
        flags += ["-Xarch_host", f]
    return flags


def _compile(src: str) -> str:
    obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
    cmd = [HIPCC, *FLAGS, *(_host_sanitizer_flags() if SANITIZE else []), "-c", os.path.join(CSRC, src),
           "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("hipcc failed for %s:\n%s\n%s" % (src, r.stdout, r.stderr))
    return obj


PROBE = os.path.join(HERE, "hbm_ceiling")
PROBE_SRC = "hbm_ceiling.hip"


def build_probe() -> str:
    """The HBM ceiling probe (a standalone program that bench.py --hbm-ceiling
    runs), next to the library."""
    tmp = PROBE + ".tmp%d" % os.getpid()
    cmd = [HIPCC, *FLAGS, os.path.join(CSRC, PROBE_SRC), "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("hipcc failed for %s:\n%s\n%s" % (PROBE_SRC, r.stdout, r.stderr))
    os.replace(tmp, PROBE)
    return PROBE


def build(verbose: bool = False) -> str:
    """Compile all sources and link libagnes.so (and the HBM ceiling probe);
    returns the library's path."""
    os.makedirs(BUILD, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=len(SOURCES)) as ex:
        objs = list(ex.map(_compile, SOURCES))
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [HIPCC, "--offload-arch=" + ARCH, "-shared", "-fPIC", "-o", tmp, *objs,
           "-L" + os.path.join(ROCM, "lib"), "-lrocprofiler-sdk-roctx", "-Wl,-rpath," + os.path.join(ROCM, "lib")]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n%s\n%s" % (r.stdout, r.stderr))
    os.replace(tmp, LIB)
    if not SANITIZE:
        build_probe()
    if verbose:
        print("built", LIB)
    return LIB


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
