"""The lemma behind the quantize kernel's reciprocal route, checked on the CPU.

For a scale with 2^-60 <= |s| <= 2^60 and a zero-point |z| <= 64 the kernel
forms w * rcp(s), corrects it with one fma residual and rounds; the claim is
that this gives the code of the correctly rounded binary32 quotient for every
bf16 weight, with any reciprocal within 2 ulp of 1/s.  quantize_route_check.c
models those binary32 steps in C and compares the codes; the run here takes
every weight pattern under about 60 scales spread over the range, and
``quantize_route_check 1 0`` (minutes) covers every scale.  The GPU tests in
test_quantize.py check the kernel itself against the oracle.
"""

import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_reciprocal_route_gives_the_division_codes(tmp_path):
    exe = str(tmp_path / "quantize_route_check")
    subprocess.run(["gcc", "-O2", "-ffp-contract=off", "-o", exe, os.path.join(HERE, "quantize_route_check.c"), "-lm"],
                   check=True)
    r = subprocess.run([exe, "509", "17"], capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stdout + r.stderr
    checks = int(r.stdout.split()[-4])
    assert checks > 10 ** 8 and " 0 mismatches" in r.stdout, r.stdout
