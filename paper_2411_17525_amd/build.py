"""Builds libhiggs.so (HIP for gfx950 + host C++) in-tree with hipcc.

usage: python -m paper_2411_17525_amd.build   (or via __graft_entry__.build())
"""
from __future__ import annotations

import concurrent.futures
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(PKG, "csrc")
ROOT = os.path.dirname(PKG)
OBJ = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libhiggs.so")

ARCH = "gfx950"
COMMON = ["-O3", "-fPIC", "-std=c++17", f"--offload-arch={ARCH}",
          "-I", os.path.join(ROOT, "include"),
          # no packed fp32 instructions in device code
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
SOURCES = {
    "higgs_abi.cpp": [],
    "grid_lloyd.cpp": ["-ffp-contract=off"],
    "bitwidth.cpp": [],
    "gptq.cpp": [],
    "rht.hip": [],
    "encode.hip": [],
    "qgemv.hip": [],
    "qgemm.hip": [],
    "scratch.hip": [],
}


def hipcc() -> str:
    path = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(path):
        raise RuntimeError("hipcc not found: the HIP toolchain is required to build libhiggs.so")
    return path


def _compile(src: str, extra: list[str], tag: str = "") -> str:
    obj = os.path.join(OBJ, src + tag + ".o")
    lang = ["-x", "hip"] if src.endswith(".hip") else []
    cmd = [hipcc(), *COMMON, *extra, *lang, "-c", os.path.join(CSRC, src), "-o", obj]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{res.stdout}\n{res.stderr}")
    return obj


# The benchmark's memory-ceiling probe: a separate library, not part of the
# product's interface.
BENCH_LIB = os.path.join(PKG, "libhiggs_bench.so")
BENCH_SOURCES = ("bench_probe.hip",)


def build_bench_probe(verbose: bool = True) -> str:
    os.makedirs(OBJ, exist_ok=True)
    objs = [_compile(src, []) for src in BENCH_SOURCES]
    tmp = BENCH_LIB + ".tmp"
    cmd = [hipcc(), "-shared", "-fPIC", f"--offload-arch={ARCH}", *objs, "-o", tmp]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"link failed: {' '.join(cmd)}\n{res.stdout}\n{res.stderr}")
    os.replace(tmp, BENCH_LIB)
    if verbose:
        print(f"built {BENCH_LIB}", file=sys.stderr)
    return BENCH_LIB


# Phase-stamp build: the library with qgemv.hip compiled with HIGGS_STAMPS
# (per-wave s_memrealtime stamps at the small-batch kernel's phase boundaries,
# read by bench.py --stamp-pass). A debug build for measurement only.
STAMP_LIB = os.path.join(PKG, "libhiggs_stamps.so")
STAMP_SOURCE = "qgemv.hip"
STAMP_FLAGS = ["-DHIGGS_STAMPS"]


def _link(objs: list[str], out: str) -> None:
    tmp = out + ".tmp"
    # rocBLAS / rocSOLVER: the library GEMM, syrk and Cholesky steps of GPTQ rounding
    cmd = [hipcc(), "-shared", "-fPIC", f"--offload-arch={ARCH}", *objs, "-o", tmp, "-lpthread",
           "-L/opt/rocm/lib", "-lrocblas", "-lrocsolver", "-Wl,-rpath,/opt/rocm/lib"]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"link failed: {' '.join(cmd)}\n{res.stdout}\n{res.stderr}")
    os.replace(tmp, out)


# Host-sanitizer build: the host C++ sources (argument validation, grids,
# bits allocation, GPTQ orchestration) compiled with AddressSanitizer and
# UndefinedBehaviorSanitizer, linked with the regular device objects (the
# GPU code is not instrumented). For the CPU tests only; load it with the
# clang ASan runtime preloaded.
SAN_DIR = os.path.join(PKG, "_build_hostsan")
SAN_LIB = os.path.join(SAN_DIR, "libhiggs.so")
HOST_SOURCES = ("higgs_abi.cpp", "grid_lloyd.cpp", "bitwidth.cpp", "gptq.cpp")
SAN_FLAGS = ["-O1", "-g", "-fno-omit-frame-pointer", "-shared-libasan",
             "-Xarch_host", "-fsanitize=address",
             "-Xarch_host", "-fsanitize=undefined",
             "-Xarch_host", "-fno-sanitize-recover=undefined"]


def build_host_sanitized(verbose: bool = True) -> str:
    os.makedirs(SAN_DIR, exist_ok=True)
    objs = []
    for src, extra in SOURCES.items():
        if src in HOST_SOURCES:
            obj = os.path.join(SAN_DIR, src + ".o")
            cmd = [hipcc(), *[f for f in COMMON if f != "-O3"], *extra, *SAN_FLAGS, "-c",
                   os.path.join(CSRC, src), "-o", obj]
            res = subprocess.run(cmd, capture_output=True, text=True)
            if res.returncode != 0:
                raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{res.stdout}\n{res.stderr}")
            objs.append(obj)
        else:
            obj = os.path.join(OBJ, src + ".o")
            if not os.path.exists(obj):
                _compile(src, extra)
            objs.append(obj)
    cmd = [hipcc(), "-shared", "-fPIC", f"--offload-arch={ARCH}", *objs, "-o", SAN_LIB,
           "-shared-libasan", "-Xarch_host", "-fsanitize=address",
           "-Xarch_host", "-fsanitize=undefined", "-lpthread", "-L/opt/rocm/lib", "-lrocblas",
           "-lrocsolver", "-Wl,-rpath,/opt/rocm/lib"]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"link failed: {' '.join(cmd)}\n{res.stdout}\n{res.stderr}")
    if verbose:
        print(f"built {SAN_LIB}", file=sys.stderr)
    return SAN_LIB


def build(verbose: bool = True) -> str:
    os.makedirs(OBJ, exist_ok=True)
    workers = min(len(SOURCES), max(1, (os.cpu_count() or 2)))
    jobs = [(src, extra, "") for src, extra in SOURCES.items()]
    jobs.append((STAMP_SOURCE, SOURCES[STAMP_SOURCE] + STAMP_FLAGS, ".stamps"))
    with concurrent.futures.ThreadPoolExecutor(workers) as ex:
        objs = list(ex.map(lambda job: _compile(*job), jobs))
    _link(objs[:len(SOURCES)], LIB)
    if verbose:
        print(f"built {LIB}", file=sys.stderr)
    stamp_objs = [objs[-1] if src == STAMP_SOURCE else o
                  for src, o in zip(SOURCES, objs[:len(SOURCES)])]
    _link(stamp_objs, STAMP_LIB)
    if verbose:
        print(f"built {STAMP_LIB}", file=sys.stderr)
    build_bench_probe(verbose)
    return LIB


if __name__ == "__main__":
    build()
