"""Pins of the streaming oracle (Sec. 4.2, cache layout and cache packing; Sec. 4.3).

* the layout against a table written out by hand from the paper's cache
  layout (anchor, retrieved, two recent chunks, current; fixed positions;
  the retrieved slot extends the recent window when nothing is admissible);
* retrieval on the test loop against the loop's construction: on the second
  lap chunk n comes back to the place of chunk n - 8, which is then the only
  admissible chunk while the ring still holds it;
* history ring residency: every chunk the layout names is still held;
* the packed keys against rotary embeddings written with Python complex
  numbers at the layout's absolute positions, and attention over the packed
  cache against attention over a cache assembled directly from them;
* correspondence on pre-pooled maps against the full-resolution definition
  (p = 2) on depth maps whose 2 x 2 blocks are constant, where pooling is
  exact.
"""

from __future__ import annotations

import cmath

import numpy as np
import pytest

from oracle import attention as OA
from oracle import reprojection as OR
from oracle.stream import StreamOracle, layout
from workloads.stream import make_stream

F = 3


@pytest.mark.parametrize("n,count,j,want", [
    (0, 0, -1, [("current", 0, 12)]),
    (1, 0, -1, [("anchor", 0, 0), ("current", 1, 12)]),
    (2, 0, -1, [("anchor", 0, 0), ("recent", 1, 9), ("current", 2, 12)]),
    (3, 0, -1, [("anchor", 0, 0), ("recent", 1, 6), ("recent", 2, 9), ("current", 3, 12)]),
    (4, 0, -1, [("anchor", 0, 0), ("extension", 1, 3), ("recent", 2, 6), ("recent", 3, 9), ("current", 4, 12)]),
    (9, 1, 1, [("anchor", 0, 0), ("retrieved", 1, 3), ("recent", 7, 6), ("recent", 8, 9), ("current", 9, 12)]),
    (30, 0, -1, [("anchor", 0, 0), ("extension", 27, 3), ("recent", 28, 6), ("recent", 29, 9), ("current", 30, 12)]),
])
def test_layout_table(n, count, j, want):
    assert layout(n, count, j, F) == want


@pytest.mark.parametrize("C", [5, 6, 10])
def test_retrieval_and_ring_on_the_loop(C):
    st = make_stream(n_chunks=14, qkv=False)
    st.L = 0
    orc = StreamOracle(st, C)
    for n in range(14):
        r = orc.step(n)
        # chunk n - 8 sits at the same place one lap earlier; it is a candidate
        # only from n = 9 on (chunk 0 is the anchor) and while the ring holds it
        resident = n - 8 >= orc.first_candidate(n)
        if n >= 9 and resident:
            assert (r["count"], r["idx"]) == (1, n - 8)
        else:
            assert r["count"] == 0
        for _, m, _ in r["parts"]:
            assert orc.ring[orc.ring_slot(m)]["chunk"] == m


def _rope(raw: np.ndarray, pos0: int, n_t: int, theta: float, hw: int) -> np.ndarray:
    """Temporal RoPE of a chunk's keys [L, T, H, D]: frame f of the chunk at position pos0 + f."""
    out = np.array(raw, np.float64, copy=True)
    L, T, H, D = raw.shape
    for l in range(L):
        for r in range(T):
            t = pos0 + r // hw
            for hh in range(H):
                for i in range(n_t):
                    z = complex(out[l, r, hh, 2 * i], out[l, r, hh, 2 * i + 1]) * cmath.exp(1j * t * theta ** (-i / n_t))
                    out[l, r, hh, 2 * i], out[l, r, hh, 2 * i + 1] = z.real, z.imag
    return out


def test_packed_cache_and_attention_against_direct_assembly():
    st = make_stream(n_chunks=11, h=2, w=3, H=1, D=16, L=1, dtype="f32")
    st.rope_t_pairs = 3
    hw, T = st.h * st.w, F * st.h * st.w
    rng = np.random.default_rng(17)
    raw = {}
    for n, ch in enumerate(st.chunks):  # keys as the network would emit them: embedded at 4F + f
        raw[n] = rng.standard_normal(ch.k.shape)
        ch.k = _rope(raw[n], 4 * F, st.rope_t_pairs, st.rope_theta, hw).astype(np.float32)
    orc = StreamOracle(st, 10)
    for n in range(11):
        r = orc.step(n)
        K = np.concatenate([_rope(raw[m], pos, st.rope_t_pairs, st.rope_theta, hw) if role != "current"
                            else st.chunks[m].k.astype(np.float64) for role, m, pos in r["parts"]], axis=1)
        V = np.concatenate([st.chunks[m].v for _, m, _ in r["parts"]], axis=1).astype(np.float64)
        np.testing.assert_allclose(r["cache_k"], K, rtol=0, atol=2e-6)
        assert np.array_equal(r["cache_v"], V.astype(np.float32))
        o, lse = OA.biased_attention(st.chunks[n].q[0].astype(np.float64), K[0], V[0], r["slot"], r["uv"], r["cidx"],
                                     st.h, st.w, st.softmax_scale, st.lam, st.sigma)
        np.testing.assert_allclose(r["o"][0], o, rtol=0, atol=2e-5)
        np.testing.assert_allclose(r["lse"][0], lse, rtol=0, atol=2e-5)
        if r["count"]:
            assert list(r["slot"][F:2 * F]) == [0, 1, 2] and (r["cidx"] >= 0).any()
        else:
            assert (r["slot"] == -1).all() and (r["cidx"] == OR.NO_SOURCE).all()


def test_pooled_correspondence_equals_full_resolution_definition():
    st = make_stream(n_chunks=12, qkv=False)
    st.L = 0
    for ch in st.chunks:  # 2 x 2 blocks of equal depth: pooling is exact
        blk = ch.depth[:, ::2, ::2]
        ch.depth = np.repeat(np.repeat(blk, 2, axis=1), 2, axis=2)
    orc = StreamOracle(st, 10)
    hits = 0
    for n in range(12):
        r = orc.step(n)
        if not r["count"]:
            continue
        src = st.chunks[r["idx"]]
        ch = st.chunks[n]
        uv, idx = OR.reproject(ch.depth, ch.c2w, ch.K, src.depth, src.c2w, src.K, st.p, st.eps)
        assert np.array_equal(idx, r["cidx"])
        assert np.array_equal(uv.view(np.uint32), r["uv"].view(np.uint32))
        hits += 1
    assert hits >= 3
