"""KV cache packing oracle (Sec. 4.2, cache layout and cache packing).

TEST INFRASTRUCTURE ONLY: like the rest of this package it may be used by
the test suite, the smoke check and the benchmark's CPU-baseline leg, never
by the library.

The clean cache of M latent frames holds an anchor chunk, the pose-retrieved
chunk(s) and a recent window (Sec. 4.2, cache layout). A retrieved chunk is
reinstated from outside the cache and placed at temporal RoPE positions
directly next to the recent window instead of its original temporal index,
so that cache positions stay in a fixed range however long the stream runs
(Sec. 4.2, cache packing). For every layer l and retrieved slot s holding
chunk j = sel[s], with T = F h w tokens per chunk:

    V_cache[l][row0 + s T + r] = V_store[l][j][r]
    K_cache[l][row0 + s T + r] = Rot(dst_pos + s F - pos[j]) K_store[l][j][r]

Readings fixed here (the paper states where the chunk goes, not how the
position embedding is laid out):

* the store keeps each historical chunk's keys and values as the cache held
  them; the keys carry the rotary position embedding (RoPE, Su et al.) of
  temporal position pos[j] + f in frame f of the chunk (pos[j] = F j, the
  chunk's original index, when no position table is given);
* RoPE acts on interleaved pairs (k_{2i}, k_{2i+1}) read as the complex
  number k_{2i} + i k_{2i+1}. The first n_t pairs carry the frame position,
  pair i with angular frequency omega_i = theta^(-i / n_t); the remaining
  pairs carry the token's grid row and column, which packing leaves alone
  (the factorised 3-D embedding of the Wan backbone the method builds on,
  temporal band first);
* moving a key from position t to t' multiplies each temporal pair by
  exp(i (t' - t) omega_i). Rotations compose, so this equals the embedding
  applied at t' to the key before any rotation;
* slot s starts at frame position dst_pos + s F: the slots are consecutive
  and the caller picks dst_pos so that they end where the recent window
  begins;
* sel[s] outside [0, n_store) leaves slot s as it was (the caller fills it,
  e.g. with the recent-window extension when no chunk is admissible);
* rotated elements are computed in float64 as x c - y s and x s + y c
  (c, s = cos, sin of delta * omega_i) and rounded once to the storage type,
  to nearest with ties to even; values and the non-temporal part of every
  key are copied bit for bit.

Arrays: bf16 tensors are passed as uint16 bit patterns, fp32 tensors as
float32; store_k / store_v are [L][n_store][T][H][D], cache_k / cache_v
[L][rows][H][D].
"""

from __future__ import annotations

import numpy as np


def rope_frequencies(n_t: int, theta: float) -> np.ndarray:
    """omega_i = theta^(-i / n_t) for the n_t temporal pairs, float64."""
    i = np.arange(n_t, dtype=np.float64)
    return np.float64(theta) ** (-(i / np.float64(n_t)))


def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    """bf16 bit patterns -> their exact float64 values."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round float64 values once to the nearest bf16, ties to even -> uint16 bits.

    bf16 keeps 8 significant bits and fp32's exponent range: at x = m 2^e
    (0.5 <= |m| < 1) consecutive bf16 numbers are 2^(e-8) apart, never less
    than the subnormal spacing 2^-133. x / spacing is exact in float64, so one
    rint (ties to even) rounds it; values past the largest bf16 become inf.
    """
    x = np.asarray(x, dtype=np.float64)
    _, e = np.frexp(x)
    q = np.maximum(e.astype(np.int64) - 8, -133)
    with np.errstate(over="ignore", invalid="ignore"):
        y = np.ldexp(np.rint(np.ldexp(x, -q)), q)
        y32 = y.astype(np.float32)  # exact for every bf16 value; 2^128 -> inf
    return (y32.view(np.uint32) >> 16).astype(np.uint16)


def rotate_temporal(k: np.ndarray, delta: int, n_t: int, theta: float) -> np.ndarray:
    """Multiply every temporal pair i < n_t of k [..., D] (float64) by exp(i delta omega_i)."""
    out = np.array(k, dtype=np.float64, copy=True)
    if n_t == 0:
        return out
    phi = np.float64(delta) * rope_frequencies(n_t, theta)
    c, s = np.cos(phi), np.sin(phi)
    x = out[..., 0:2 * n_t:2].copy()
    y = out[..., 1:2 * n_t:2].copy()
    out[..., 0:2 * n_t:2] = x * c - y * s
    out[..., 1:2 * n_t:2] = x * s + y * c
    return out


def pack_retrieved_kv(store_k, store_v, store_pos, sel, dst_pos, cache_k, cache_v, dst_row0, F, n_t, theta):
    """Packed copies of cache_k and cache_v (see the module docstring)."""
    store_k = np.asarray(store_k)
    store_v = np.asarray(store_v)
    bf16 = store_k.dtype == np.uint16
    ck = np.array(cache_k, copy=True)
    cv = np.array(cache_v, copy=True)
    n_store, T = store_k.shape[1], store_k.shape[2]
    for s, j in enumerate(np.asarray(sel).tolist()):
        if not 0 <= j < n_store:
            continue
        pos_j = F * j if store_pos is None else int(store_pos[j])
        delta = int(dst_pos) + s * F - pos_j
        rows = slice(dst_row0 + s * T, dst_row0 + (s + 1) * T)
        cv[:, rows] = store_v[:, j]
        src = store_k[:, j]
        ck[:, rows] = src
        if n_t > 0:
            k64 = bf16_to_f64(src) if bf16 else src.astype(np.float64)
            r = rotate_temporal(k64, delta, n_t, theta)[..., :2 * n_t]
            ck[:, rows, :, :2 * n_t] = round_bf16(r) if bf16 else r.astype(np.float32)
    return ck, cv
