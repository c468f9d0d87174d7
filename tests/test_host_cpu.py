"""Host-side contracts that need no GPU.

* bench.py refuses more than one GPU with a message and a non-zero status
  before touching a device, reads the power state amd-smi prints (or
  records none where amd-smi is missing), and builds every key of its
  one-line JSON result (headline, roofline and CPU-baseline objects);
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


_SMI_TEXT = """GPU: 0
    POWER:
        SOCKET_POWER: 1350 W
        GFX_VOLTAGE: N/A
        MEM_VOLTAGE: N/A
    CLOCK:
        GFX_0:
            CLK: 1800 MHz
            MAX_CLK: 2400 MHz
        GFX_1:
            CLK: 1700 MHz
            MAX_CLK: 2400 MHz
        MEM_0:
            CLK: 2000 MHz
    TEMPERATURE:
        EDGE: N/A
        HOTSPOT: 60 °C
        MEM: 45 °C
"""


def test_bench_result_carries_every_key():
    """The keys of the JSON line, found among the string keys of the dict
    literals and subscript assignments that bench.py builds."""
    import ast

    tree = ast.parse(open(os.path.join(ROOT, "bench.py")).read())
    keys = set()
    for node in ast.walk(tree):
        if isinstance(node, ast.Dict):
            keys |= {k.value for k in node.keys if isinstance(k, ast.Constant) and isinstance(k.value, str)}
        elif isinstance(node, ast.Subscript) and isinstance(node.ctx, ast.Store):
            if isinstance(node.slice, ast.Constant) and isinstance(node.slice.value, str):
                keys.add(node.slice.value)
    headline = {"metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "higher_is_better", "scaling",
                "vs_baseline", "dtype", "data", "config", "workload"}
    roofline = {"roofline", "bound", "achieved", "peak", "frac", "traffic"}
    baseline = {"cpu_baseline", "cores", "kind", "sample"}
    missing = (headline | roofline | baseline) - keys
    assert not missing, f"bench.py never builds {sorted(missing)}"


def test_bench_power_state_reads_amd_smi(monkeypatch):
    sys.path.insert(0, ROOT)
    import bench
    import torch

    class Done:
        stdout = _SMI_TEXT

    monkeypatch.setattr(torch.cuda, "synchronize", lambda *a, **k: None)
    monkeypatch.setattr(subprocess, "run", lambda *a, **k: Done())
    ps = bench._power_state(lambda: None, secs=0.3, settle_s=0.0)
    assert ps is not None and ps["samples"] >= 1
    # the clock is the mean over the XCDs; MAX_CLK and the HBM clock are not read as XCD clocks
    assert (ps["socket_power_w"], ps["gfx_clock_mhz"], ps["hotspot_c"], ps["hbm_c"]) == (1350.0, 1750.0, 60.0, 45.0)

    def missing(*a, **k):
        raise FileNotFoundError("amd-smi")

    monkeypatch.setattr(subprocess, "run", missing)
    assert bench._power_state(lambda: None, secs=0.2, settle_s=0.0) is None


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
