"""Pins of the KV cache packing oracle (Sec. 4.2, cache layout and cache packing).

Each pin checks the oracle against something other than itself:

* bf16 rounding against torch's fp32 -> bf16 conversion (a library routine,
  round to nearest even) on fp32-representable inputs, and against exact
  rational rounding (fractions.Fraction) on float64 inputs, where a double
  rounding through fp32 would differ;
* the rotation against RoPE written with Python complex numbers at absolute
  positions: moving a key embedded at t1 to t2 must give the key embedded at
  t2 (the defining property of the re-rotation), plus its invariants
  (identity at delta 0, composition, pair norms, untouched spatial band);
* the gather against a pure-Python loop over slots, tokens, heads and pairs.
"""

from __future__ import annotations

import cmath
import math
from fractions import Fraction

import numpy as np
import pytest
import torch

from oracle import kvpack as K
from workloads.synth import bf16_bits


# ----------------------------------------------------------------------------
# rounding to bf16


def _bits_of_f32(x: np.ndarray) -> np.ndarray:
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def test_round_bf16_matches_torch_on_fp32_values():
    rng = np.random.default_rng(7)
    parts = [
        rng.standard_normal(20000).astype(np.float32),
        (rng.standard_normal(5000) * 1e30).astype(np.float32),
        (rng.standard_normal(5000) * 1e-30).astype(np.float32),
        # fp32 subnormals and the bf16 subnormal range
        (rng.standard_normal(5000) * 1e-39).astype(np.float32),
        (rng.integers(1, 1 << 23, 5000).astype(np.uint32)).view(np.float32),
        # exact halfway points between neighbouring bf16 numbers
        ((rng.integers(0x00800000, 0x7f000000, 5000).astype(np.uint32) & 0xffff0000) | 0x8000).view(np.float32),
        np.array([0.0, -0.0, 1.0, -1.0, 3.3895314e38, -3.3895314e38], dtype=np.float32),
    ]
    x = np.concatenate(parts)
    got = K.round_bf16(x.astype(np.float64))
    want = _bits_of_f32(x)
    assert np.array_equal(got, want)


@pytest.mark.parametrize(
    "x, bits",
    [
        (1 + 2.0**-8, 0x3F80),  # tie -> even (1.0)
        (1 + 3 * 2.0**-8, 0x3F82),  # tie -> even (1 + 2^-6)
        (1 + 2.0**-8 + 2.0**-40, 0x3F81),  # just above the tie: one rounding goes up
        (-(1 + 2.0**-8 + 2.0**-40), 0xBF81),
        (2.0**-134, 0x0000),  # half the smallest subnormal: tie -> 0
        (3 * 2.0**-134, 0x0002),  # tie between subnormals 1 and 2 -> 2
        (2.0**-134 + 2.0**-160, 0x0001),
        ((2 - 2.0**-8) * 2.0**127, 0x7F80),  # halfway to 2^128 -> inf
        ((2 - 2.0**-8) * 2.0**127 - 2.0**90, 0x7F7F),  # largest finite bf16
        (-0.0, 0x8000),
    ],
)
def test_round_bf16_hand_cases(x, bits):
    assert int(K.round_bf16(np.array([x]))[0]) == bits


def _round_bf16_exact(x: float) -> int:
    """Nearest bf16 to x (ties to even) by exact rational arithmetic -> bits."""
    if x == 0.0:
        return 0x8000 if math.copysign(1.0, x) < 0 else 0
    fx = Fraction(x)
    sign = 0x8000 if fx < 0 else 0
    a = abs(fx)
    # spacing of bf16 numbers around a: 2^(e-8) for a in [2^(e-1), 2^e), at least 2^-133
    e = math.frexp(abs(x))[1]
    spacing = Fraction(2) ** max(e - 8, -133)
    n = a / spacing
    lo = math.floor(n)
    rem = n - lo
    m = lo + 1 if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and lo % 2 == 1) else lo
    val = m * spacing
    if val >= Fraction(2) ** 128:
        return sign | 0x7F80
    f32 = np.float32(float(val))
    assert Fraction(float(f32)) == val
    return sign | (int(np.array([f32]).view(np.uint32)[0]) >> 16)


def test_round_bf16_matches_exact_rational_rounding():
    rng = np.random.default_rng(11)
    x = np.concatenate([
        rng.standard_normal(3000),
        rng.standard_normal(500) * 1e-38,
        rng.standard_normal(500) * 1e37,
        # float64 values within 2^-30 (relative) of a bf16 halfway point
        (np.round(rng.standard_normal(1000) * 2**8) / 2**8 + 2.0**-9) * (1 + rng.uniform(-2**-30, 2**-30, 1000)),
    ])
    got = K.round_bf16(x)
    want = np.array([_round_bf16_exact(float(v)) for v in x], dtype=np.uint16)
    assert np.array_equal(got, want)


# ----------------------------------------------------------------------------
# rotation of the temporal band


def test_frequencies_closed_form():
    w = K.rope_frequencies(22, 10000.0)
    assert w[0] == 1.0
    assert abs(w[11] - 0.01) <= 2 * np.spacing(0.01)  # 10000^(-1/2)
    assert np.all(np.diff(w) < 0)
    for i in range(22):
        assert abs(w[i] - math.pow(10000.0, -i / 22)) <= np.spacing(w[i])


def _rope_at(k: np.ndarray, t: int, n_t: int, theta: float) -> np.ndarray:
    """Temporal RoPE at absolute position t, pair by pair with Python complex numbers."""
    out = np.array(k, dtype=np.float64, copy=True)
    flat = out.reshape(-1, out.shape[-1])
    for row in flat:
        for i in range(n_t):
            z = complex(row[2 * i], row[2 * i + 1]) * cmath.exp(1j * t * theta ** (-i / n_t))
            row[2 * i], row[2 * i + 1] = z.real, z.imag
    return out


@pytest.mark.parametrize("t1, t2", [(0, 5), (600, 6), (7, -3), (123456, 9)])
def test_rotation_moves_embedding_between_positions(t1, t2):
    rng = np.random.default_rng(t1 + 3)
    raw = rng.standard_normal((4, 3, 64))
    n_t, theta = 11, 10000.0
    at_t1 = _rope_at(raw, t1, n_t, theta)
    moved = K.rotate_temporal(at_t1, t2 - t1, n_t, theta)
    np.testing.assert_allclose(moved, _rope_at(raw, t2, n_t, theta), rtol=0, atol=1e-9)


def test_rotation_invariants():
    rng = np.random.default_rng(5)
    k = rng.standard_normal((6, 128))
    n_t, theta = 22, 10000.0
    assert np.array_equal(K.rotate_temporal(k, 0, n_t, theta), k)
    ab = K.rotate_temporal(K.rotate_temporal(k, 17, n_t, theta), -40, n_t, theta)
    np.testing.assert_allclose(ab, K.rotate_temporal(k, -23, n_t, theta), rtol=0, atol=1e-12)
    r = K.rotate_temporal(k, 1234, n_t, theta)
    norms = lambda a: np.hypot(a[:, 0:2 * n_t:2], a[:, 1:2 * n_t:2])
    np.testing.assert_allclose(norms(r), norms(k), rtol=1e-14)
    assert np.array_equal(r[:, 2 * n_t:], k[:, 2 * n_t:])
    # pair 0 has omega = 1: (1, 0) turns by delta radians
    e = np.zeros((1, 128)); e[0, 0] = 1.0
    r1 = K.rotate_temporal(e, 1, n_t, theta)
    assert r1[0, 0] == math.cos(1.0) and r1[0, 1] == math.sin(1.0)


# ----------------------------------------------------------------------------
# gather into the packed slots


def _pack_brute(store_k, store_v, store_pos, sel, dst_pos, cache_k, cache_v, row0, F, n_t, theta):
    ck = np.array(cache_k, copy=True)
    cv = np.array(cache_v, copy=True)
    L, n_store, T, H, D = store_k.shape
    bf16 = store_k.dtype == np.uint16
    val = (lambda b: float(np.array([int(b) << 16], dtype=np.uint32).view(np.float32)[0])) if bf16 else float
    for s, j in enumerate(sel):
        if j < 0 or j >= n_store:
            continue
        delta = dst_pos + s * F - (F * j if store_pos is None else int(store_pos[j]))
        for l in range(L):
            for r in range(T):
                for hh in range(H):
                    dst = row0 + s * T + r
                    cv[l, dst, hh] = store_v[l, j, r, hh]
                    ck[l, dst, hh] = store_k[l, j, r, hh]
                    for i in range(n_t):
                        z = complex(val(store_k[l, j, r, hh, 2 * i]), val(store_k[l, j, r, hh, 2 * i + 1]))
                        z = z * cmath.exp(1j * (delta * theta ** (-i / n_t)))
                        if bf16:
                            ck[l, dst, hh, 2 * i] = _round_bf16_exact(z.real)
                            ck[l, dst, hh, 2 * i + 1] = _round_bf16_exact(z.imag)
                        else:
                            ck[l, dst, hh, 2 * i] = np.float32(z.real)
                            ck[l, dst, hh, 2 * i + 1] = np.float32(z.imag)
    return ck, cv


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("with_pos", [False, True])
def test_pack_matches_loop_version(dtype, with_pos):
    rng = np.random.default_rng(3 if with_pos else 4)
    L, n_store, F, hw, H, D, n_t, theta = 2, 5, 2, 3, 2, 16, 3, 10000.0
    T = F * hw
    raw_k = rng.standard_normal((L, n_store, T, H, D)).astype(np.float32)
    raw_v = rng.standard_normal((L, n_store, T, H, D)).astype(np.float32)
    rows = 5 * T + 2
    if dtype == "bf16":
        sk, sv = bf16_bits(raw_k), bf16_bits(raw_v)
        ck0 = np.full((L, rows, H, D), 0x7FC1, np.uint16)
        cv0 = np.full((L, rows, H, D), 0x7FC2, np.uint16)
    else:
        sk, sv = raw_k, raw_v
        ck0 = np.full((L, rows, H, D), np.nan, np.float32)
        cv0 = np.full((L, rows, H, D), -7.0, np.float32)
    pos = rng.integers(-50, 500, n_store).astype(np.int32) if with_pos else None
    sel = [3, -1, 0, 3, 9]  # a repeat, an empty slot and one out of range
    args = (sk, sv, pos, sel, 40, ck0, cv0, 2, F, n_t, theta)
    gk, gv = K.pack_retrieved_kv(*args)
    wk, wv = _pack_brute(*args)
    assert gk.tobytes() == wk.tobytes()
    assert gv.tobytes() == wv.tobytes()
    # untouched: the two leading rows and the slots whose selection is empty or out of range
    for s in (1, 4):
        sl = slice(2 + s * T, 2 + (s + 1) * T)
        assert gk[:, sl].tobytes() == ck0[:, sl].tobytes()
        assert gv[:, sl].tobytes() == cv0[:, sl].tobytes()
    assert gk[:, :2].tobytes() == ck0[:, :2].tobytes()


def test_pack_places_chunks_next_to_recent_window():
    """Keys stored with RoPE at their original frame positions come out embedded
    at the packed positions, up to one rounding (the reading of Sec. 4.2)."""
    rng = np.random.default_rng(9)
    L, n_store, F, hw, H, D, n_t, theta = 1, 8, 3, 2, 1, 32, 6, 10000.0
    T = F * hw
    raw = rng.standard_normal((L, n_store, T, H, D))
    frame_of_row = np.arange(T) // hw
    stored = np.empty_like(raw)
    for j in range(n_store):
        for r in range(T):
            stored[0, j, r] = _rope_at(raw[0, j, r], F * j + frame_of_row[r], n_t, theta)
    sk = stored.astype(np.float32)
    # cache: anchor (F frames) | 2 retrieved slots | recent window starting at frame 3F
    recent_start, sel = 3 * F, [6, 2]
    ck0 = np.zeros((L, 5 * T, H, D), np.float32)
    gk, _ = K.pack_retrieved_kv(sk, sk, None, sel, recent_start - len(sel) * F, ck0, ck0, T, F, n_t, theta)
    for s, j in enumerate(sel):
        for r in range(T):
            want = _rope_at(sk[0, j, r].astype(np.float64), F + s * F + frame_of_row[r] - (F * j + frame_of_row[r]), n_t, theta)
            want_direct = _rope_at(raw[0, j, r], F + s * F + frame_of_row[r], n_t, theta)
            got = gk[0, T + s * T + r].astype(np.float64)
            np.testing.assert_allclose(got, want, rtol=0, atol=4e-7)
            np.testing.assert_allclose(got, want_direct, rtol=0, atol=4e-6)
