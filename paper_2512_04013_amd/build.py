"""Build libaug.so in-tree for gfx950.

HIP sources are compiled by hipcc for gfx950 only; the host-only C++ sources
(planner, batch former, status strings) by the same compiler as plain C++
without FMA contraction, so the former's double-precision arithmetic is
reproducible. Objects go to ``_build/`` next to this file; the library lands
in this package directory.

    python -m paper_2512_04013_amd.build
"""

from __future__ import annotations

import concurrent.futures as cf
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(PKG, "_build")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libaug.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

HIP_SOURCES = ["attn.hip", "kvappend.hip", "kvpark.hip", "upload.hip"]
CPP_SOURCES = ["plan.cpp", "former.cpp", "status.cpp"]

COMMON = ["-O3", "-std=c++17", "-fPIC", f"-I{INCLUDE}", f"-I{CSRC}", "-Wall", "-Wno-unused-function"]
HIP_FLAGS = ["--offload-arch=gfx950", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             "-mcumode"]
CPP_FLAGS = ["-x", "c++", "-ffp-contract=off", "-fno-fast-math"]


def _compile(src: str, verbose: bool) -> str:
    obj = os.path.join(BUILD, os.path.basename(src) + ".o")
    path = os.path.join(CSRC, src)
    if src.endswith(".hip"):
        cmd = [HIPCC, *COMMON, *HIP_FLAGS, "-c", path, "-o", obj]
    else:
        cmd = [HIPCC, *COMMON, *CPP_FLAGS, "-c", path, "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    out = (r.stdout + r.stderr).strip()
    # hipcc's host pass does not know the packed-fp32 target feature; that note is harmless
    out = "\n".join(ln for ln in out.splitlines() if "packed-fp32-ops" not in ln)
    if r.returncode != 0:
        raise RuntimeError(f"compile of {src} failed:\n{out}")
    if out and verbose:
        print(out, flush=True)
    return obj


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    srcs = HIP_SOURCES + CPP_SOURCES
    with cf.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        objs = list(ex.map(lambda s: _compile(s, verbose), srcs))
    tmp = LIB + ".tmp"
    cmd = [HIPCC, "-shared", "-fPIC", "--offload-arch=gfx950", *objs, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}{r.stderr}")
    os.replace(tmp, LIB)
    return LIB


HOST_SAN_LIB = os.path.join(BUILD, "libaug_host_san.so")


def build_host_sanitized(verbose: bool = False) -> str:
    """The host-only sources (planner, batch former, status strings) built by
    g++ with AddressSanitizer and UndefinedBehaviorSanitizer into
    ``_build/libaug_host_san.so``, for CPU test runs of the host code under the
    sanitizers (the process must preload the compiler's libasan). The library
    has no device entry points."""
    os.makedirs(BUILD, exist_ok=True)
    srcs = [os.path.join(CSRC, s) for s in CPP_SOURCES]
    tmp = HOST_SAN_LIB + ".tmp"
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fPIC", "-shared", f"-I{INCLUDE}", f"-I{CSRC}",
           "-ffp-contract=off", "-fno-fast-math", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all", *srcs, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"sanitized host build failed:\n{r.stdout}{r.stderr}")
    os.replace(tmp, HOST_SAN_LIB)
    return HOST_SAN_LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
