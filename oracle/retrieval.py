"""Pose retrieval oracle (Sec. 4.2, "Loop-closure retrieval", Eq. retrieval).

For the current chunk n with camera centre c_n and unit viewing direction
v_n, each historical chunk j gets the score

    s(j) = |c_j - c_n|_2 / E + w_v (1 - v_j . v_n)

and is admissible when all three gates hold: |c_j - c_n|_2 / E <= tau_c,
v_j . v_n >= cos(tau_v) and n - j >= Delta. The method reinstates the
admissible chunk of smallest score; an empty admissible set leaves the
retrieved slot to the recent window.

Readings fixed here (the paper is silent on them):

* a pose is a row-major 4x4 camera-to-world matrix; the centre is its last
  column and the viewing direction is R e_z, the third column of R, used as
  stored (not renormalised);
* bank entry j is chunk j; entries below ``first_candidate`` are skipped
  (the anchor chunk is already resident in the cache);
* the top-k generalisation returns the k admissible chunks of smallest
  score, ties broken by smaller j; fewer than k admissible -> count < k and
  the unused outputs are -1;
* cos(tau_v) is evaluated once in double precision with the C library's
  ``cos`` (``math.cos``), on tau_v as the fp32 value the interface carries.

Arithmetic: all inputs are converted to float64 and every operation is one
IEEE double operation in the order written below (no fused multiply-add).
"""

from __future__ import annotations

import math

import numpy as np


def centre_and_view(c2w: np.ndarray):
    """(c, v) of poses [..., 4, 4]: c = last column, v = R e_z (third column)."""
    m = np.asarray(c2w, dtype=np.float64)
    return m[..., :3, 3], m[..., :3, 2]


def scores(bank_c2w, query_c2w, E, w_v):
    """Distance term d(j), alignment a(j) = v_j . v_n and score s(j) for one
    query pose against every bank pose (Eq. retrieval, first line).

    Returns three float64 arrays of shape [N]."""
    cj, vj = centre_and_view(bank_c2w)
    cn, vn = centre_and_view(query_c2w)
    E = np.float64(np.float32(E))
    w_v = np.float64(np.float32(w_v))
    dx = cj[:, 0] - cn[0]
    dy = cj[:, 1] - cn[1]
    dz = cj[:, 2] - cn[2]
    d = np.sqrt(dx * dx + dy * dy + dz * dz) / E
    a = vj[:, 0] * vn[0] + vj[:, 1] * vn[1] + vj[:, 2] * vn[2]
    s = d + w_v * (1.0 - a)
    return d, a, s


def admissible(d, a, j, n, tau_c, tau_v, delta, first_candidate):
    """The admissible set A_n (Eq. retrieval, second line) as a mask."""
    tau_c = np.float64(np.float32(tau_c))
    cos_tv = math.cos(float(np.float32(tau_v)))
    return (j >= first_candidate) & (n - j >= delta) & (d <= tau_c) & (a >= cos_tv)


def retrieve(bank_c2w, query_c2w, query_chunk, E, w_v, tau_c, tau_v, delta, first_candidate, k):
    """Top-k pose retrieval for every query.

    Returns (idx [Q, k] int32 padded with -1, score [Q, k] float64 padded with
    +inf, count [Q] int32)."""
    bank_c2w = np.asarray(bank_c2w)
    query_c2w = np.asarray(query_c2w)
    Q = query_c2w.shape[0]
    N = bank_c2w.shape[0]
    j = np.arange(N, dtype=np.int64)
    idx = np.full((Q, k), -1, np.int32)
    sc = np.full((Q, k), np.inf)
    count = np.zeros(Q, np.int32)
    for qi in range(Q):
        n = int(query_chunk[qi])
        d, a, s = scores(bank_c2w, query_c2w[qi], E, w_v)
        ok = admissible(d, a, j, n, tau_c, tau_v, delta, first_candidate)
        cand = j[ok]
        order = np.lexsort((cand, s[ok]))  # primary key s, then j
        take = cand[order][:k]
        idx[qi, : len(take)] = take
        sc[qi, : len(take)] = s[take]
        count[qi] = len(take)
    return idx, sc, count


def frame_selection(idx, count, frames_per_chunk):
    """Expand retrieved chunk ids to the frames they contribute, in order:
    entry i*F + f is frame idx[i]*F + f, or -1 where i >= count."""
    Q, k = idx.shape
    F = frames_per_chunk
    sel = np.full((Q, k * F), -1, np.int32)
    for qi in range(Q):
        for i in range(int(count[qi])):
            for f in range(F):
                sel[qi, i * F + f] = idx[qi, i] * F + f
    return sel


def near_ties(bank_c2w, query_c2w, query_chunk, E, w_v, tau_c, tau_v, delta, first_candidate, k,
              rel=1e-12):
    """Diagnostics: per query, whether the k-th and (k+1)-th admissible
    scores are within ``rel`` (relative) of each other, and how many gate
    margins lie within ``rel`` of their thresholds. Both should be zero on
    generic inputs; the parity tests report them."""
    ties = 0
    margins = 0
    N = bank_c2w.shape[0]
    j = np.arange(N)
    tc = np.float64(np.float32(tau_c))
    ctv = math.cos(float(np.float32(tau_v)))
    for qi in range(query_c2w.shape[0]):
        n = int(query_chunk[qi])
        d, a, s = scores(bank_c2w, query_c2w[qi], E, w_v)
        ok = admissible(d, a, j, n, tau_c, tau_v, delta, first_candidate)
        ss = np.sort(s[ok])
        if len(ss) > k and abs(ss[k] - ss[k - 1]) < rel * max(1.0, abs(ss[k])):
            ties += 1
        live = (j >= first_candidate) & (n - j >= delta)
        margins += int(np.sum(live & (np.abs(d - tc) < rel * max(1.0, tc))))
        margins += int(np.sum(live & (np.abs(a - ctv) < rel)))
    return ties, margins
