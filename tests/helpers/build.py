"""Build the GPU test helper librngprobe.so (gfx950) next to its source.

    python tests/helpers/build.py

The helper includes the library's rng.hpp and is compiled with the flags the
library uses for the translation units that draw random numbers, so that the
values it returns are the ones the library's kernels compute.
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
CSRC = os.path.join(ROOT, "paper_2606_03928_amd", "csrc")
LIB = os.path.join(HERE, "librngprobe.so")


def build() -> str:
    sys.path.insert(0, ROOT)
    from paper_2606_03928_amd.build import hipcc, ARCH
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [hipcc(), "-x", "hip", "--offload-arch=" + ARCH, "-O3", "-std=c++17", "-fPIC", "-shared",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", "-ffp-contract=off",
           "-I", CSRC, os.path.join(HERE, "rng_probe.hip"), "-o", tmp]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError("building librngprobe.so failed:\n" + res.stderr)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build())
