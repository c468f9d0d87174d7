"""GPU pin of the bf16 / fp8 kernel's bias geometry (Sec. 4.3, Eq. bias):
the bias is the only thing the logits of retrieved frames depend on, and V
reads the softmax weights out, so the comparison with the fp64 oracle can
use a relative bar derived from the kernel's bf16 roundings (tests/bias_pin.py
states the case and the bar; tests/test_bias_pin_power.py shows on the CPU
that a half-cell u^ shift, an x/y swap, key centres without the +1/2, and a
10 % sigma or lambda error each fail it). Run on the 30 x 52 and 45 x 80 token
grids, with tiles straddling retrieved and unbiased frames, 20 retrieved
frames (past the 16 the bf16 kernel stages in LDS), key parts 1 and 4, bf16
and fp8 logits."""

from __future__ import annotations

import numpy as np
import pytest
import torch

import paper_2607_21848_amd as rv
from tests import bias_pin as BP
from tests.gpu_helpers import dev, host
from workloads.synth import fp8e4m3_bits

pytestmark = pytest.mark.gpu

_REF = {}


def _case(name):
    if name not in _REF:
        case = BP.make_case(**BP.CASES[name])
        _REF[name] = (case, BP.oracle(case))
    return _REF[name]


@pytest.mark.parametrize("parts", [1, 4])
@pytest.mark.parametrize("dtype", ["bf16", "fp8"])
@pytest.mark.parametrize("name", sorted(BP.CASES))
def test_bias_geometry(name, dtype, parts):
    case, (O_ref, LSE_ref) = _case(name)
    print(f"bias geometry {name} {dtype} key_parts={parts}", flush=True)
    if dtype == "bf16":
        q, k = dev(case["q"], torch.bfloat16), dev(case["k"], torch.bfloat16)
    else:
        q = torch.from_numpy(fp8e4m3_bits(case["q"])).cuda().view(torch.float8_e4m3fn)
        k = torch.from_numpy(fp8e4m3_bits(case["k"])).cuda().view(torch.float8_e4m3fn)
    v = dev(case["v"], torch.bfloat16)
    o, lse = rv.biased_chunk_attention(q, k, v, dev(case["slot"]), dev(case["uv"]), dev(case["idx"]), h=case["h"],
                                       w=case["w"], softmax_scale=case["scale"], lam=case["lam"],
                                       sigma=case["sigma"], key_parts=parts)
    torch.cuda.synchronize()
    ok, ratio, lerr = BP.compare(host(o), host(lse).T, O_ref, LSE_ref.T)
    print(f"  worst |dO| / bar = {ratio:.3f} (bar {BP.O_REL_BAR:.4f} |O| + {BP.O_ABS_BAR:g}), "
          f"max |dLSE| = {lerr:.3e} (bar {BP.LSE_BAR:g})")
    assert ok
