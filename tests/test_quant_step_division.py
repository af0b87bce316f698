"""The quantiser's step size Delta = Range / (2^b - 1) (Eq. 6) is formed on the
GPU from the product with the rounded reciprocal and one fma correction
instead of a divide.  That is the correctly rounded quotient for every finite
Range >= 0 at the three supported widths; this checks it over all 2^31 such
binary32 values on the host (IEEE arithmetic, no contraction)."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))


def test_step_division_is_correctly_rounded(tmp_path):
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no C compiler")
    exe = str(tmp_path / "div_by_levels")
    # -march=native for hardware fma; the result does not depend on it
    flags = ["-O3", "-ffp-contract=off", "-fno-fast-math"]
    r = subprocess.run([cc, *flags, "-march=native", "-o", exe,
                        os.path.join(HERE, "helpers", "div_by_levels.c"), "-lm"], capture_output=True)
    if r.returncode != 0:
        subprocess.run([cc, *flags, "-o", exe, os.path.join(HERE, "helpers", "div_by_levels.c"),
                        "-lm"], check=True, capture_output=True)
    out = subprocess.run([exe], check=True, capture_output=True, text=True, timeout=600).stdout
    got = {line.split()[0]: int(line.split()[1]) for line in out.strip().splitlines()}
    assert got == {"3": 0, "15": 0, "255": 0}
