"""Host sanitizer builds (CPU only): the oracle and the C ABI's host-side code.

* The oracle (oracle/vase_oracle.c) with gcc -fsanitize=address,undefined,
  driven by tests/helpers/sanitize_oracle.c over every entry point on small and
  boundary shapes.
* libvase's host code (argument validation, workspace sizing, dispatch) with
  AddressSanitizer and UBSan (hipcc -Xarch_host, device code unchanged), driven
  by tests/helpers/sanitize_abi.cpp: every entry point with arguments the
  validation must reject, so nothing reaches a device, and workspace sizes over
  the accepted range.
Either run stops at the first report (-fno-sanitize-recover=all).
"""
import concurrent.futures as cf
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HELP = os.path.join(ROOT, "tests", "helpers")
CSRC = os.path.join(ROOT, "paper_2606_03928_amd", "csrc")
SAN_HOST = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-sanitize-recover=all"]


def _run(cmd, env=None, timeout=600):
    res = subprocess.run(cmd, capture_output=True, text=True, env=env, timeout=timeout)
    assert res.returncode == 0, "%s\n%s\n%s" % (" ".join(cmd), res.stdout[-3000:], res.stderr[-3000:])
    return res.stdout


def test_oracle_under_asan_ubsan(tmp_path):
    exe = str(tmp_path / "san_oracle")
    _run(["gcc", "-O1", "-g", "-std=c11", "-fopenmp", "-ffp-contract=off", "-fno-fast-math",
          "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-Wall",
          os.path.join(HELP, "sanitize_oracle.c"), os.path.join(ROOT, "oracle", "vase_oracle.c"),
          "-lm", "-o", exe])
    env = dict(os.environ, OMP_NUM_THREADS="2", ASAN_OPTIONS="detect_leaks=1")
    assert _run([exe], env=env).strip().endswith("ok")


@pytest.mark.skipif(shutil.which("hipcc") is None and not os.path.exists("/opt/rocm/bin/hipcc"),
                    reason="hipcc is needed to build the library's host code")
def test_abi_host_code_under_asan_ubsan(tmp_path):
    from paper_2606_03928_amd.build import SOURCES, ARCH, hipcc
    base = [hipcc(), "-x", "hip", "--offload-arch=" + ARCH, "-O1", "-g", "-std=c++17", "-fPIC",
            "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"] + SAN_HOST + [
            "-I", os.path.join(ROOT, "include"), "-I", CSRC]

    def compile_one(src):
        obj = str(tmp_path / (os.path.basename(src) + ".o"))
        extra = ["-ffp-contract=off"] if os.path.basename(src) in ("select.hip", "dkv.hip",
                                                                     "quant.hip") else []
        _run(base + extra + ["-c", src, "-o", obj])
        return obj

    srcs = [os.path.join(CSRC, s) for s in SOURCES] + [os.path.join(HELP, "sanitize_abi.cpp")]
    with cf.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        objs = list(ex.map(compile_one, srcs))
    exe = str(tmp_path / "san_abi")
    _run([hipcc(), "--offload-arch=" + ARCH] + SAN_HOST + objs + ["-o", exe])
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0")   # the HIP runtime keeps its own allocations
    assert "ok" in _run([exe], env=env)
