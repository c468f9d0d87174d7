"""Pure-Python loop versions of the three stages, for tiny inputs only.

They restate the same definitions as the vectorised oracle with scalar
Python floats, explicit loops and ``math.fsum`` / ``math.exp``, and serve to
pin it: a slip in the vectorised indexing, broadcasting or masking shows up
as a disagreement here.

* ``retrieve``       -- Sec. 4.2, Eq. retrieval (exhaustive: score every
  chunk, keep admissible ones, full sort by (score, index));
* ``reproject``      -- Sec. 4.3, Eq. reprojection / Eq. visibility, one
  token at a time through 3x3 matrix products written as explicit sums;
* ``attention_row``  -- Sec. 4.3, Eq. bias, one query row: logits, bias,
  softmax normalised with ``math.fsum``.
"""

from __future__ import annotations

import math


def _col(m, c):
    return [float(m[r][c]) for r in range(3)]


def retrieve(bank_c2w, query_c2w, n, E, w_v, tau_c, tau_v, delta, first_candidate, k):
    """Returns (list of chunk ids, list of scores) for one query."""
    E, w_v, tau_c, tau_v = (float(x) for x in (E, w_v, tau_c, tau_v))
    cn, vn = _col(query_c2w, 3), _col(query_c2w, 2)
    cands = []
    for j in range(len(bank_c2w)):
        cj, vj = _col(bank_c2w[j], 3), _col(bank_c2w[j], 2)
        dist = math.sqrt(sum((cj[i] - cn[i]) ** 2 for i in range(3))) / E
        align = sum(vj[i] * vn[i] for i in range(3))
        if j < first_candidate or n - j < delta:
            continue
        if dist > tau_c or align < math.cos(tau_v):
            continue
        cands.append((dist + w_v * (1.0 - align), j))
    cands.sort()
    top = cands[:k]
    return [j for _, j in top], [s for s, _ in top]


def _pool(depth, i, j, p):
    return sum(float(depth[p * i + a][p * j + b]) for a in range(p) for b in range(p)) / (p * p)


def reproject(tgt_depth, tgt_c2w, tgt_K, src_depth, src_c2w, src_K, p, eps):
    """One target frame into one source frame. Returns a list of
    (uhx, uhy, idx) per token in row-major order (uh = None when not
    computed)."""
    Hd, Wd = len(tgt_depth), len(tgt_depth[0])
    h, w = Hd // p, Wd // p
    fxt, fyt, cxt, cyt = (float(x) / p for x in tgt_K)
    fxs, fys, cxs, cys = (float(x) / p for x in src_K)
    Rt = [[float(tgt_c2w[r][c]) for c in range(3)] for r in range(3)]
    Rs = [[float(src_c2w[r][c]) for c in range(3)] for r in range(3)]
    ct, cs = _col(tgt_c2w, 3), _col(src_c2w, 3)
    out = []
    for i in range(h):
        for j in range(w):
            z = _pool(tgt_depth, i, j, p)
            if not (math.isfinite(z) and z > 0):
                out.append((None, None, -1))
                continue
            ray = [(j + 0.5 - cxt) / fxt, (i + 0.5 - cyt) / fyt, 1.0]
            Xt = [z * r for r in ray]
            world = [sum(Rt[r][c] * Xt[c] for c in range(3)) + ct[r] for r in range(3)]
            rel = [world[r] - cs[r] for r in range(3)]
            Xs = [sum(Rs[c][r] * rel[c] for c in range(3)) for r in range(3)]  # R_s^T rel
            if not Xs[2] > 0:
                out.append((None, None, -2))
                continue
            uhx = (fxs * Xs[0] + cxs * Xs[2]) / Xs[2]
            uhy = (fys * Xs[1] + cys * Xs[2]) / Xs[2]
            if not (0 <= uhx < w and 0 <= uhy < h):
                out.append((uhx, uhy, -3))
                continue
            kx, ky = int(math.floor(uhx)), int(math.floor(uhy))
            Ds = _pool(src_depth, ky, kx, p)
            if Xs[2] <= (1.0 + float(eps)) * Ds:
                out.append((uhx, uhy, ky * w + kx))
            else:
                out.append((uhx, uhy, -4))
    return out


def attention_row(qrow, keys, vals, col_info, scale, lam, sigma):
    """One query row of one head.

    qrow: list of D floats; keys, vals: lists of Lk rows; col_info[k] is
    None (unbiased column) or (kx, ky, uhx, uhy) for a biased one. Returns
    (output row, lse)."""
    D = len(qrow)
    logits = []
    for kk in range(len(keys)):
        a = math.fsum(qrow[d] * keys[kk][d] for d in range(D)) * scale
        info = col_info[kk]
        if info is not None:
            kx, ky, uhx, uhy = info
            dist2 = (kx + 0.5 - uhx) ** 2 + (ky + 0.5 - uhy) ** 2
            a += lam * (-dist2 / (2.0 * sigma * sigma))
        logits.append(a)
    m = max(logits)
    ex = [math.exp(a - m) for a in logits]
    den = math.fsum(ex)
    out = [math.fsum(ex[kk] * vals[kk][d] for kk in range(len(keys))) / den for d in range(D)]
    return out, m + math.log(den)
