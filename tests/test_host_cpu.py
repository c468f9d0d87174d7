"""Host-side contracts that need no GPU.

* bench.py refuses more than one GPU with a message and a non-zero status
  before touching a device;
* the entry module exposes build() and smoke();
* the product path never reaches the oracle: importing the package loads
  nothing from oracle/, and no package source refers to it;
* without the built library every entry point raises (there is no CPU path).
"""

from __future__ import annotations

import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2607_21848_amd")


def test_bench_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 2
    assert "one GPU" in r.stdout


def test_entry_module_exposes_build_and_smoke():
    import __graft_entry__ as g
    assert callable(g.build) and callable(g.smoke)


def test_package_import_does_not_load_the_oracle():
    code = "import sys, paper_2607_21848_amd; print(any(m == 'oracle' or m.startswith('oracle.') for m in sys.modules))"
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 0, r.stderr
    assert r.stdout.strip() == "False"


def test_package_sources_never_refer_to_the_oracle():
    for dirpath, _, files in os.walk(PKG):
        for f in files:
            if f.endswith((".py", ".hip", ".cpp", ".h")):
                with open(os.path.join(dirpath, f)) as fh:
                    text = fh.read()
                assert "import oracle" not in text and "from oracle" not in text, f


def test_missing_library_raises(monkeypatch):
    from paper_2607_21848_amd import _lib
    monkeypatch.setattr(_lib, "_LIB", None)
    monkeypatch.setattr(_lib, "LIB_PATH", os.path.join(ROOT, "no-such-dir", "librevisit.so"))
    with pytest.raises(RuntimeError, match="no CPU fallback"):
        _lib.lib()
