"""Build libvase.so (HIP, gfx950 only) in-tree.

    python -m paper_2606_03928_amd.build

Every translation unit is compiled with hipcc for gfx950 with packed-fp32 code
generation disabled; select.hip, dkv.hip and quant.hip additionally with
-ffp-contract=off (their random numbers and quantisation codes are fixed IEEE
binary32 operation sequences).
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD_DIR = os.path.join(ROOT, "_build")
LIB_PATH = os.path.join(PKG, "libvase.so")
# measurement probes for the benchmark's roofline denominators (not part of the round)
PEAKS_SOURCE = "peaks.hip"
PEAKS_PATH = os.path.join(PKG, "libvase_peaks.so")

SOURCES = ["abi.hip", "score.hip", "select.hip", "compact.hip", "decode.hip", "dkv.hip",
           "quant.hip", "order.hip"]
HEADERS = ["vase_internal.hpp"]
ARCH = "gfx950"


def hipcc() -> str:
    p = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(p):
        raise RuntimeError("hipcc not found: the HIP library cannot be built")
    return p


def _flags(src: str):
    f = ["-x", "hip", "--offload-arch=" + ARCH, "-O3", "-std=c++17", "-fPIC",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-Wall", "-Wno-unused-function", "-I", INCLUDE, "-I", CSRC]
    if src in ("select.hip", "dkv.hip", "quant.hip"):
        f.append("-ffp-contract=off")
    return f


def _compile(src: str, verbose: bool) -> str:
    obj = os.path.join(BUILD_DIR, src.replace(".hip", ".o"))
    cmd = [hipcc()] + _flags(src) + ["-c", os.path.join(CSRC, src), "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    # the host pass does not know the packed-fp32 target feature; that warning is harmless
    noise = "'-packed-fp32-ops' is not a recognized feature"
    err = "\n".join(l for l in res.stderr.splitlines() if noise not in l)
    if res.returncode != 0:
        raise RuntimeError("compiling %s failed:\n%s" % (src, err))
    if verbose and err.strip():
        print(err, file=sys.stderr)
    return obj


def build(verbose: bool = False) -> str:
    """Compile every source and link libvase.so; returns its path."""
    os.makedirs(BUILD_DIR, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=min(len(SOURCES), 8)) as ex:
        objs = list(ex.map(lambda s: _compile(s, verbose), SOURCES))
    tmp = LIB_PATH + ".tmp%d" % os.getpid()
    cmd = [hipcc(), "--offload-arch=" + ARCH, "-shared", "-fPIC", "-o", tmp] + objs
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError("linking libvase.so failed:\n" + res.stderr)
    os.replace(tmp, LIB_PATH)
    build_peaks(verbose)
    return LIB_PATH


def build_peaks(verbose: bool = False) -> str:
    """Compile the benchmark's peak probes into libvase_peaks.so."""
    tmp = PEAKS_PATH + ".tmp%d" % os.getpid()
    cmd = [hipcc()] + _flags(PEAKS_SOURCE) + ["-shared", os.path.join(CSRC, PEAKS_SOURCE), "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError("building libvase_peaks.so failed:\n" + res.stderr)
    os.replace(tmp, PEAKS_PATH)
    return PEAKS_PATH


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
