"""Builds, in-tree, libcpattn.so (the attention step: HIP kernels + C ABI,
gfx950, hipcc), libcplayer.so (the element-wise kernels of the decoder layer
around it, gfx950), libcppeaks.so (peak-rate microbenchmarks, gfx950) and
libcpsched.so (the host scheduler, plain C++17, g++)."""

from __future__ import annotations

import concurrent.futures as cf
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libcpattn.so")
SCHED_LIB = os.path.join(PKG, "libcpsched.so")
LAYER_LIB = os.path.join(PKG, "libcplayer.so")
LAYER_SOURCES = ["layer.hip", "gemm.hip"]
PEAKS_LIB = os.path.join(PKG, "libcppeaks.so")
PEAKS_SOURCES = ["peaks.hip"]
CXX = os.environ.get("CXX", "g++")
SOURCES = ["api.hip", "plan.cpp", "append.hip", "decode.hip", "prefill.hip", "merge.hip"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-Wall",
    # packed fp32 VALU forms are kept out of the generated code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", os.path.join(ROOT, "include"), "-I", CSRC,
]


def _compile(src: str) -> str:
    obj = os.path.join(BUILD, os.path.basename(src) + ".o")
    lang = ["-x", "hip"] if src.endswith(".hip") else []
    cmd = [HIPCC, *FLAGS, *lang, "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n{r.stderr}")
    if r.stderr.strip():
        sys.stderr.write(r.stderr)
    return obj


def build(jobs: int = 8) -> str:
    os.makedirs(BUILD, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=jobs) as ex:
        objs = list(ex.map(_compile, SOURCES + LAYER_SOURCES + PEAKS_SOURCES))
    n1, n2 = len(SOURCES), len(SOURCES) + len(LAYER_SOURCES)
    _link(objs[:n1], LIB)
    _link(objs[n1:n2], LAYER_LIB)
    _link(objs[n2:], PEAKS_LIB)
    build_sched()
    return LIB


def _link(objs, out):
    tmp = out + ".tmp"
    r = subprocess.run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", tmp],
                       capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link of {os.path.basename(out)} failed:\n{r.stderr}")
    os.replace(tmp, out)


def build_sched() -> str:
    tmp = SCHED_LIB + ".tmp"
    cmd = [CXX, "-O3", "-std=c++17", "-fPIC", "-shared", "-Wall", "-Wextra",
           "-I", os.path.join(ROOT, "include"), os.path.join(CSRC, "sched.cpp"), "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"{CXX} failed on sched.cpp:\n{r.stderr}")
    os.replace(tmp, SCHED_LIB)
    return SCHED_LIB


if __name__ == "__main__":
    print(build())
