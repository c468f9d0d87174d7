"""Biased chunk attention oracle (Sec. 4.3, Eq. bias; design choices (ii), (iii)).

For a query token p and a key token k lying in a retrieved (source) frame s,

    B_s(p, k) = - |u_k - u^_s(p)|^2 / (2 sigma^2)
    A_pk      = q_p . k_k / sqrt(d) + lambda B_s(p, k)

and every other logit is the plain scaled dot product. The output is
O = softmax_k(A) V per head, with LSE_p = log sum_k exp(A_pk) (natural log).

Readings fixed here:

* only key columns whose KV frame carries a retrieved-frame slot s >= 0
  are biased (design choice (ii)); the anchor, recent and current frames
  are not;
* a query whose correspondence into frame s was rejected (idx < 0) gets no
  bias on frame s's columns (design choice (iii), per source frame);
* u_k is the key's token centre (k_x + 1/2, k_y + 1/2) with
  (k_y, k_x) = divmod(k mod (h w), w); u^ is the continuous reprojected
  position (Eq. bias uses it, not the snapped cell);
* the bias is added after the 1/sqrt(d) scaling, and is not itself scaled;
  ``softmax_scale`` is the caller's 1/sqrt(d);
* no mask: every query attends to all Lk keys (bidirectional chunk).

All arithmetic is float64; query rows are processed in blocks so that full
sizes fit in memory, and ``rows`` restricts the computation to sampled
query rows.
"""

from __future__ import annotations

import numpy as np


def fp8e4m3_values(bits: np.ndarray) -> np.ndarray:
    """Exact float64 values of fp8 e4m3 codes (OCP: sign, 4 exponent bits with
    bias 7, 3 mantissa bits; exponent 0 subnormal; 0x7f / 0xff NaN)."""
    b = np.asarray(bits, dtype=np.uint8).astype(np.int64)
    sign = np.where(b & 0x80, -1.0, 1.0)
    e = (b >> 3) & 0xF
    m = (b & 0x7).astype(np.float64)
    mag = np.where(e == 0, np.ldexp(m / 8.0, -6), np.ldexp(1.0 + m / 8.0, e - 7))
    mag = np.where((e == 15) & (m == 7), np.nan, mag)
    return sign * mag


def key_centres(Lk, h, w):
    """Token-grid centres (x, y) of every key column: [Lk, 2] float64."""
    t = np.arange(Lk) % (h * w)
    ky, kx = np.divmod(t, w)
    return np.stack([kx + 0.5, ky + 0.5], axis=-1).astype(np.float64)


def bias_block(rows, Lk, h, w, slot, corr_uv, corr_idx, sigma):
    """B[rows, :] per Eq. bias (zero where no bias applies): [len(rows), Lk]."""
    rows = np.asarray(rows)
    B = np.zeros((len(rows), Lk))
    if corr_idx is None or len(slot) == 0:
        return B
    kc = key_centres(Lk, h, w)
    hw = h * w
    two_s2 = 2.0 * np.float64(np.float32(sigma)) ** 2
    for f, s in enumerate(np.asarray(slot)):
        if s < 0:
            continue
        cols = slice(f * hw, (f + 1) * hw)
        uh = np.asarray(corr_uv[s], dtype=np.float64)[rows]  # [R, 2]
        ok = np.asarray(corr_idx[s])[rows] >= 0
        dx = kc[cols, 0][None, :] - uh[:, 0:1]
        dy = kc[cols, 1][None, :] - uh[:, 1:2]
        b = -(dx * dx + dy * dy) / two_s2
        B[:, cols] = np.where(ok[:, None], b, 0.0)
    return B


def biased_attention(q, k, v, slot, corr_uv, corr_idx, h, w, softmax_scale, lam, sigma,
                     rows=None, heads=None, block=256):
    """O and LSE for the given query rows and heads.

    q: [Lq, H, D], k, v: [Lk, H, D] (any float dtype; converted to float64).
    slot: [Lk / (h w)] int; corr_uv: [S, Lq, 2]; corr_idx: [S, Lq] (or None).
    Returns O [len(rows), len(heads), D] float64 and LSE [len(heads), len(rows)].
    """
    Lq, H, D = q.shape
    Lk = k.shape[0]
    rows = np.arange(Lq) if rows is None else np.asarray(rows)
    heads = np.arange(H) if heads is None else np.asarray(heads)
    scale = np.float64(np.float32(softmax_scale))
    lam = np.float64(np.float32(lam))
    O = np.zeros((len(rows), len(heads), D))
    LSE = np.zeros((len(heads), len(rows)))
    for r0 in range(0, len(rows), block):
        rr = rows[r0:r0 + block]
        B = bias_block(rr, Lk, h, w, slot, corr_uv, corr_idx, sigma) if lam != 0.0 else None
        for hi, hd in enumerate(heads):
            Q = np.asarray(q[rr, hd, :], dtype=np.float64)
            Kh = np.asarray(k[:, hd, :], dtype=np.float64)
            Vh = np.asarray(v[:, hd, :], dtype=np.float64)
            A = (Q @ Kh.T) * scale
            if B is not None:
                A = A + lam * B
            m = A.max(axis=1, keepdims=True)
            E = np.exp(A - m)
            den = E.sum(axis=1, keepdims=True)
            O[r0:r0 + len(rr), hi, :] = (E @ Vh) / den
            LSE[hi, r0:r0 + len(rr)] = (m + np.log(den))[:, 0]
    return O, LSE
