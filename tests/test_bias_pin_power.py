"""The bias-geometry bar has power (Sec. 4.3, Eq. bias): on the cases the GPU
pin runs, the oracle with a planted mistake fails the bar against the oracle
itself, for every mistake, and the correct oracle passes it trivially. Also
checks that the case is what its docstring says (q, k, v exact in bf16 and
fp8 e4m3; one-hot columns read weights)."""

from __future__ import annotations

import numpy as np
import pytest

from tests import bias_pin as BP
import workloads as W
from workloads.synth import fp8e4m3_bits


@pytest.fixture(scope="module", params=sorted(BP.CASES))
def case_and_ref(request):
    spec = dict(BP.CASES[request.param])
    # smaller query sets keep the CPU suite short; the geometry is the same
    spec["Lq"] = 24
    case = BP.make_case(**spec)
    return request.param, case, BP.oracle(case)


def test_case_values_exact_in_bf16_and_fp8(case_and_ref):
    _, c, _ = case_and_ref
    for name in ("q", "k", "v"):
        x = c[name]
        assert np.array_equal(W.bf16_round(x), x), name
    from oracle.attention import fp8e4m3_values
    for name in ("q", "k"):
        x = c[name]
        assert np.array_equal(fp8e4m3_values(fp8e4m3_bits(x)), x.astype(np.float64)), name


def test_one_hot_columns_read_softmax_weights(case_and_ref):
    """O columns 0..111 are the weights of the block keys: they sum with the
    rest of the frame's keys to the frame's mass column."""
    _, c, (O, LSE) = case_and_ref
    assert np.all(O[:, :, :112] >= 0) and np.all(O[:, :, :112] <= 1)
    # all frame-indicator columns together hold the whole mass
    assert np.allclose(O[:, :, 112:].sum(axis=-1), 1.0, atol=1e-12)
    # the block holds the bulk of its frame's Gaussian, so a share of the row
    # near 1 / (retrieved frames), less where rejected frames carry weight 1 per key
    assert np.median(O[:, :, :112].sum(axis=-1)) > 0.005


def test_correct_oracle_passes(case_and_ref):
    _, _, (O, LSE) = case_and_ref
    ok, ratio, lerr = BP.compare(O, LSE, O, LSE)
    assert ok and ratio == 0.0 and lerr == 0.0


def test_planted_mistakes_fail_the_bar(case_and_ref):
    name, case, (O, LSE) = case_and_ref
    for mistake, Om, Lm in BP.planted_mistakes(case):
        ok, ratio, lerr = BP.compare(Om, Lm, O, LSE)
        print(f"{name}: {mistake}: worst |dO|/bar = {ratio:.1f}, max |dLSE| = {lerr:.3e}")
        assert not ok, f"{name}: the bar does not see '{mistake}'"
        # by a clear margin, not at the edge of the bar
        assert ratio > 3.0 or lerr > 3 * BP.LSE_BAR, mistake
