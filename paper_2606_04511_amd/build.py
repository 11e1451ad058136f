"""Build libsparda.so for gfx950 with hipcc (in-tree, no torch extension machinery).

Each translation unit is compiled to an object under ``_build/`` and linked into
``paper_2606_04511_amd/libsparda.so``; the benchmark's microbenchmarks go into
``paper_2606_04511_amd/libsparda_peaks.so``.  Every HIP object is built with packed-FP32 instruction
selection turned off (``-Xclang -target-feature -Xclang -packed-fp32-ops``).
"""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libsparda.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

# Microbenchmarks of the hardware limits, for the benchmark only (not part of the C ABI).
PEAKS_SOURCE = "peaks.hip"
PEAKS_LIB = os.path.join(PKG, "libsparda_peaks.so")

SOURCES = ["compress.hip", "select.hip", "select_prefill.hip", "score_max.hip", "select_multihead.hip", "indexer_kl.hip", "attention.hip", "attention_prefill.hip", "gather.hip", "sparda_abi.cpp"]

COMMON = ["-O3", "-std=c++17", "-fPIC", "--offload-arch=gfx950", "-I", os.path.join(ROOT, "include"), "-I", CSRC,
          "-Wall", "-Wno-unused-function"]
NO_PACKED_FP32 = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def _compile(src: str) -> str:
    obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
    cmd = [HIPCC, *COMMON, *NO_PACKED_FP32, "-x", "hip", "-c", os.path.join(CSRC, src), "-o", obj]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{res.stdout}\n{res.stderr}")
    warn = "\n".join(l for l in res.stderr.splitlines() if "packed-fp32-ops" not in l and l.strip())
    if warn:
        sys.stderr.write(warn + "\n")
    return obj


def _link(objs, lib: str) -> None:
    tmp = lib + ".tmp%d" % os.getpid()
    cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp, *objs]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"link failed:\n{res.stdout}\n{res.stderr}")
    os.replace(tmp, lib)


def build() -> str:
    os.makedirs(BUILD, exist_ok=True)
    with ThreadPoolExecutor(max_workers=min(len(SOURCES) + 1, os.cpu_count() or 4)) as ex:
        objs = list(ex.map(_compile, SOURCES + [PEAKS_SOURCE]))
    _link(objs[:-1], LIB)
    _link(objs[-1:], PEAKS_LIB)
    return LIB


if __name__ == "__main__":
    print(build())
