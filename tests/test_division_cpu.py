"""The shared-reciprocal quotient of the correspondence kernel
(paper_2607_21848_amd/csrc/quotient.h, Markstein's correction step) against
IEEE division on the CPU: the same header built for the host with
contraction off and the C library's correctly rounded fma, over operands in
the ranges the configurations produce, log-uniform operands over
[2^-500, 2^500], adversarial significands next to 1 and 2 with quotients at
binade edges, and random significands. Every quotient must be bit-identical
(tests/division/quotient_check.cpp)."""

import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))


@pytest.fixture(scope="module")
def checker(tmp_path_factory):
    cxx = shutil.which("g++") or shutil.which("c++")
    if cxx is None:
        pytest.skip("no host C++ compiler")
    exe = str(tmp_path_factory.mktemp("quotient") / "quotient_check")
    subprocess.run([cxx, "-std=c++17", "-O2", "-ffp-contract=off", os.path.join(HERE, "division", "quotient_check.cpp"),
                    "-o", exe, "-lm"], check=True)
    return exe


def test_shared_reciprocal_quotient_is_ieee_division(checker):
    r = subprocess.run([checker, "1000000"], capture_output=True, text=True)
    print(r.stdout, r.stderr)
    assert r.returncode == 0
    assert "mismatches config 0, wide 0, hard 0, random 0" in r.stdout
