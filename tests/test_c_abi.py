"""The C interface from plain C (tests/c_abi/abi_check.c, gcc, C11): the
header compiles as C, every entry point is callable without C++ or Python,
host-side validation rejects bad arguments before any device call, and on a
GPU both correspondence calls map every token onto itself for identical
poses (Sec. 4.3)."""

from __future__ import annotations

import os
import shutil
import subprocess

import pytest

from tests.c_abi import build_check

pytestmark = pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not available")


def _exe() -> str:
    if not os.path.exists(os.path.join(build_check.LIBDIR, "librevisit.so")):
        pytest.fail("librevisit.so is not built: run `python -m paper_2607_21848_amd.build`")
    if build_check.stale():
        build_check.build()
    return build_check.EXE


def test_c_abi_host_checks():
    r = subprocess.run([_exe()], capture_output=True, text=True, timeout=60)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "abi_check: ok" in r.stdout


@pytest.mark.gpu
def test_c_abi_identity_on_the_device():
    import torch

    if torch.cuda.device_count() == 0:  # counts devices without initialising one
        pytest.skip("no GPU")
    print("abi_check --gpu: identity correspondence from plain C", flush=True)
    r = subprocess.run([_exe(), "--gpu"], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "abi_check: ok" in r.stdout
