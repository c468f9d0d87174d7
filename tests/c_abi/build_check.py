"""Build tests/c_abi/abi_check (a plain-C consumer of librevisit) with gcc as C11."""

from __future__ import annotations

import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
SRC = os.path.join(HERE, "abi_check.c")
EXE = os.path.join(HERE, "abi_check")
LIBDIR = os.path.join(ROOT, "paper_2607_21848_amd")
HEADER = os.path.join(ROOT, "include", "revisit.h")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def stale() -> bool:
    if not os.path.exists(EXE):
        return True
    inputs = [SRC, HEADER, os.path.join(LIBDIR, "librevisit.so")]
    return os.path.getmtime(EXE) < max(os.path.getmtime(p) for p in inputs if os.path.exists(p))


def build() -> str:
    cmd = ["gcc", "-std=c11", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(ROOT, "include"), "-I", os.path.join(ROCM, "include"), SRC, "-o", EXE,
           "-L", LIBDIR, "-lrevisit", "-L", os.path.join(ROCM, "lib"), "-lamdhip64",
           f"-Wl,-rpath,{LIBDIR}", f"-Wl,-rpath,{os.path.join(ROCM, 'lib')}"]
    subprocess.run(cmd, check=True)
    return EXE
