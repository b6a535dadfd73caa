"""Builds libmx.so (the gfx950 HIP library behind include/mx.h) in-tree with hipcc."""
from __future__ import annotations

import concurrent.futures as cf
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(ROOT, "_build", "mx")
LIB = os.path.join(PKG, "libmx.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

SOURCES = ["mx_abi.cpp", "elementwise.hip", "attention.hip", "gemm.hip"]
FLAGS = ["--offload-arch=gfx950", "-O3", "-fPIC", "-std=c++17", "-fvisibility=hidden",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-Wno-unused-command-line-argument", "-I", os.path.join(ROOT, "include"), "-I", CSRC]


# Host-side AddressSanitizer (the host code only: the flags reach the host
# compilation pass alone, device code is built as usual).
ASAN_HOST = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fno-omit-frame-pointer"]


def _compile(src: str, verbose: bool, build_dir: str = BUILD, extra=()) -> str:
    obj = os.path.join(build_dir, os.path.splitext(src)[0] + ".o")
    cmd = [HIPCC] + FLAGS + list(extra) + ["-x", "hip", "-c", os.path.join(CSRC, src), "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    err = "\n".join(l for l in res.stderr.splitlines() if "packed-fp32-ops" not in l)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n{err}")
    if err.strip() and verbose:
        print(err)
    return obj


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=min(8, len(SOURCES))) as ex:
        objs = list(ex.map(lambda s: _compile(s, verbose), SOURCES))
    tmp = LIB + ".tmp"
    # -z defs: an undefined symbol fails the build, not the first load
    cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-Wl,-z,defs", "-o", tmp] + objs
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


def build_asan_host(verbose: bool = False) -> str:
    """A copy of the library whose host code (argument checks, planning,
    metadata packing) runs under AddressSanitizer: _build/asan/libmx.so.
    Load it with MX_LIB_PATH set to that file and the sanitizer runtime
    preloaded (see the test notes)."""
    build_dir = os.path.join(ROOT, "_build", "asan")
    os.makedirs(build_dir, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=min(8, len(SOURCES))) as ex:
        objs = list(ex.map(lambda s: _compile(s, verbose, build_dir,
                                              ASAN_HOST if s.endswith(".cpp") else ()), SOURCES))
    out = os.path.join(build_dir, "libmx.so")
    cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-Xarch_host",
           "-fsanitize=address", "-shared-libasan", "-o", out] + objs
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    return out


def device_asm(src: str, out: str) -> str:
    """gfx950 assembly of one library source, compiled with the library's flags."""
    cmd = [HIPCC] + FLAGS + ["-x", "hip", "--cuda-device-only", "-S",
                             os.path.join(CSRC, src), "-o", out]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc -S failed on {src}:\n{res.stderr}")
    return out


def build_workload_gen(verbose: bool = False) -> str:
    """The device-side input generator (workload/libmxgen.so)."""
    src = os.path.join(ROOT, "workload", "csrc", "mxgen.hip")
    out = os.path.join(ROOT, "workload", "libmxgen.so")
    cmd = [HIPCC] + FLAGS[:-4] + ["-shared", "-o", out + ".tmp", src]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed on mxgen.hip:\n{res.stderr}")
    os.replace(out + ".tmp", out)
    return out


if __name__ == "__main__":
    if "--asan-host" in sys.argv:
        print(build_asan_host(verbose="-v" in sys.argv))
    else:
        print(build(verbose="-v" in sys.argv))
        print(build_workload_gen(verbose="-v" in sys.argv))
