"""Streaming oracle: the paper's cache layout run chunk by chunk (Sec. 4.2,
cache layout, loop-closure retrieval and cache packing; Sec. 4.3).

TEST INFRASTRUCTURE ONLY: like the rest of this package it may be used by
the test suite, the smoke check and the benchmark's CPU-baseline leg, never
by the library. It composes the pinned oracles of this package (retrieval,
reprojection, kvpack, attention) in the order the method runs them.

Readings fixed here:

* Cache layout (M = 4F clean frames): the anchor is chunk 0, then one
  retrieved chunk, then the recent window of the two chunks before the
  current one. Chunk n attends over [anchor | retrieved | recent n-2 |
  recent n-1 | current n], each part present only when it exists. Chunk 0
  attends to itself, and the anchor is never also a recent chunk.
* Positions are fixed per role, so the cache stays in a fixed position range
  however long the stream runs:
  - anchor at frames 0..F-1;
  - retrieved at F..2F-1, directly before the recent window;
  - recent at 2F..4F-1;
  - current at 4F..5F-1.
  Every chunk is generated in the current role, so its keys are stored with
  the rotary embedding of position 4F + f.
* Retrieval (Eq. retrieval) takes k = 1. It runs over the representative
  poses (middle frame) of the chunks before n that the history ring still
  holds, with the anchor excluded.
* When no chunk is admissible, the retrieved slot extends the recent window.
  It holds chunk n-3 (if n-3 >= 1), without bias. Before n = 4 nothing can go
  there and the slot is left out.
* The history ring keeps the anchor and the C - 1 newest chunks. Chunk m >= 1
  lives at ring slot 1 + (m - 1) mod (C - 1). Chunk n enters the ring at the
  start of its own step (the gap gate keeps it from being a candidate), so
  chunks n - C + 2 .. n are resident during step n. C >= 5 keeps chunk n-3
  resident.
* Per chunk the ring keeps:
  - the pre-pooled token depth (p x p mean rounded to fp32);
  - the frame poses;
  - the token-grid intrinsics K / p (fp32);
  - every layer's keys and values.
* Correspondence (Sec. 4.3) maps the current chunk's tokens into the
  retrieved chunk's F frames on the pooled maps (p = 1). Without a retrieved
  chunk every code is "no source" (-5).
* Attention (Eq. bias) runs per layer over the packed cache. The retrieved
  frames carry slots 0..F-1 when a chunk was retrieved; every other frame,
  including an extension chunk, carries -1.
"""

from __future__ import annotations

import numpy as np

from . import attention as OA
from . import kvpack as OK
from . import reprojection as OR
from . import retrieval as ORT


def layout(n: int, count: int, j: int, F: int):
    """Parts of chunk n's attention range: (role, chunk, first frame position)."""
    parts = []
    if n >= 1:
        parts.append(("anchor", 0, 0))
    if n >= 4:
        parts.append(("retrieved", j, F) if count > 0 else ("extension", n - 3, F))
    if n - 2 >= 1:
        parts.append(("recent", n - 2, 2 * F))
    if n - 1 >= 1:
        parts.append(("recent", n - 1, 3 * F))
    parts.append(("current", n, 4 * F))
    return parts


class StreamOracle:
    def __init__(self, stream, capacity: int):
        if capacity < 5:
            raise ValueError("the history ring needs at least 5 chunks")
        self.st = stream
        self.C = capacity
        self.bank = []  # representative pose of every chunk so far (chunk id = index)
        self.ring = {}  # ring slot -> the chunk's stored data

    def ring_slot(self, m: int) -> int:
        return 0 if m == 0 else 1 + (m - 1) % (self.C - 1)

    def first_candidate(self, n: int) -> int:
        return max(1, n - self.C + 2)

    def _values(self, a):
        return OK.bf16_to_f64(a) if self.st.dtype == "bf16" else np.asarray(a, np.float64)

    def step(self, n: int, rows=None):
        st = self.st
        F, h, w, p = st.F, st.h, st.w, st.p
        T = F * h * w
        ch = st.chunks[n]
        # the chunk enters the history ring and the pose bank
        pooled = OR.pooled_depth(ch.depth, p).astype(np.float32)
        tok_K = (np.asarray(ch.K, np.float64) / p).astype(np.float32)
        self.ring[self.ring_slot(n)] = dict(chunk=n, depth=pooled, c2w=ch.c2w, K=tok_K, k=ch.k, v=ch.v)
        self.bank.append(ch.c2w[F // 2])
        # retrieval over the resident history
        if n > 0:
            idx, _, cnt = ORT.retrieve(np.stack(self.bank[:n]), ch.c2w[F // 2][None], np.array([n]), st.E, st.w_v,
                                       st.tau_c, st.tau_v, st.delta, self.first_candidate(n), 1)
            count, j = int(cnt[0]), int(idx[0, 0])
        else:
            count, j = 0, -1
        parts = layout(n, count, j, F)
        for _, m, _ in parts:
            assert self.ring[self.ring_slot(m)]["chunk"] == m, "layout names a chunk the ring no longer holds"
        # the packed cache, every layer; positions fixed per role
        Lk = T * len(parts)
        stor = np.uint16 if st.dtype == "bf16" else np.float32
        ck = np.zeros((st.L, Lk, st.H, st.D), stor)
        cv = np.zeros((st.L, Lk, st.H, st.D), stor)
        slot = np.full(Lk // (h * w), -1, np.int32)
        for i, (role, m, pos) in enumerate(parts):
            r = self.ring[self.ring_slot(m)]
            if st.L > 0:
                n_t = 0 if role == "current" else st.rope_t_pairs
                ck, cv = OK.pack_retrieved_kv(r["k"][:, None], r["v"][:, None], np.array([4 * F]), [0], pos, ck, cv,
                                              i * T, F, n_t, st.rope_theta)
            if role == "retrieved":
                slot[i * F:(i + 1) * F] = np.arange(F)
        # correspondence of the current tokens into the retrieved chunk's frames
        if count > 0:
            src = self.ring[self.ring_slot(j)]
            uv, cidx = OR.reproject(pooled, ch.c2w, tok_K, src["depth"], src["c2w"], src["K"], 1, st.eps)
        else:
            uv = np.full((F, T, 2), np.nan, np.float32)
            cidx = np.full((F, T), OR.NO_SOURCE, np.int32)
        # biased attention of every layer
        O, LSE = [], []
        for l in range(st.L):
            o, lse = OA.biased_attention(self._values(ch.q[l]), self._values(ck[l]), self._values(cv[l]), slot, uv,
                                         cidx, h, w, st.softmax_scale, st.lam, st.sigma, rows=rows)
            O.append(o)
            LSE.append(lse)
        return dict(count=count, idx=j, parts=parts, slot=slot, uv=uv, cidx=cidx, cache_k=ck, cache_v=cv,
                    o=np.stack(O) if O else None, lse=np.stack(LSE) if LSE else None)
