"""MI355X (gfx950) hot path of training-free revisit consistency
(arXiv 2607.21848, Sec. 4.2 and Sec. 4.3).

Python binding of librevisit: argument marshalling only. Every stage runs
in the library's HIP kernels; torch tensors supply device memory and the
current HIP stream. The entry points mirror include/revisit.h:

* ``retrieve_chunks``          -- pose retrieval (Sec. 4.2, Eq. retrieval)
* ``reproject_correspondence`` -- depth/pose reprojection and visibility
                                  (Sec. 4.3, Eq. reprojection, Eq. visibility)
* ``reproject_rotation``       -- its fixed-centre case, the rotation / zoom
                                  homography without depth (Sec. 4.3)
* ``biased_chunk_attention``   -- attention with the Gaussian correspondence
                                  bias (Sec. 4.3, Eq. bias)

Each accepts optional preallocated outputs (``out=``) and, where a kernel
needs scratch memory, a preallocated ``workspace=`` (a uint8 GPU tensor of at
least ``attention_workspace_size(...)`` / ``retrieve_workspace_size(...)``
bytes), so a caller can run the path without allocating; without one the
binding allocates the workspace with torch on the current stream.
"""

from __future__ import annotations

import ctypes
from typing import Optional, Sequence

import torch

from . import _lib
from ._lib import BF16, F32, FP8_QK, MAX_K, RevisitError, last_error, lib, status_string  # noqa: F401

__all__ = ["retrieve_chunks", "reproject_correspondence", "reproject_rotation", "biased_chunk_attention", "pack_retrieved_kv",
           "pool_token_depth", "StreamDriver", "attention_workspace_size", "retrieve_workspace_size",
           "RevisitError", "lib"]


def _ptr(t: Optional[torch.Tensor]):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else ctypes.c_void_p(0)


def _stream(device: torch.device):
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _need(t: torch.Tensor, name: str, dtype: torch.dtype, shape: Optional[Sequence[int]] = None, device=None):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be a GPU tensor (got {t.device}); there is no CPU path")
    if device is not None and t.device != device:
        raise ValueError(f"{name} is on {t.device}, expected {device}")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype} (got {t.dtype})")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    return t


def _workspace(nbytes: int, workspace: Optional[torch.Tensor], dev: torch.device, name: str):
    """The caller's workspace (checked) or a fresh one of nbytes; None when nothing is needed."""
    if workspace is not None:
        _need(workspace, name, torch.uint8, None, dev)
        return workspace
    if nbytes == 0:
        return None
    return torch.empty(nbytes, dtype=torch.uint8, device=dev)


def retrieve_workspace_size(n_bank: int, n_query: int, k: int) -> int:
    """Bytes of workspace retrieve_chunks needs (0 for banks of at most 8192 entries)."""
    n = ctypes.c_size_t(0)
    _lib.check("rc_retrieve_workspace_size", lib().rc_retrieve_workspace_size(int(n_bank), int(n_query), int(k),
                                                                              ctypes.byref(n)))
    return int(n.value)


def attention_workspace_size(dtype: torch.dtype, Lq: int, Lk: int, H: int, D: int, key_parts: int = 0) -> int:
    """Bytes of workspace biased_chunk_attention needs on the current device
    (dtype: torch.bfloat16, torch.float32 or torch.float8_e4m3fn for q)."""
    n = ctypes.c_size_t(0)
    _lib.check("rc_attention_workspace_size",
               lib().rc_attention_workspace_size(_attn_dtype(dtype), int(Lq), int(Lk), int(H), int(D), int(key_parts),
                                                 ctypes.byref(n)))
    return int(n.value)


def _attn_dtype(dtype: torch.dtype) -> int:
    if dtype == torch.bfloat16:
        return BF16
    if dtype == torch.float32:
        return F32
    if dtype == torch.float8_e4m3fn:
        return FP8_QK
    raise TypeError(f"q must be bfloat16, float32 or float8_e4m3fn (got {dtype})")


def retrieve_chunks(bank_c2w: torch.Tensor, query_c2w: torch.Tensor, query_chunk: torch.Tensor, *,
                    E: float, w_v: float, tau_c: float, tau_v: float, delta: int, first_candidate: int, k: int,
                    frames_per_chunk: Optional[int] = None, out=None, workspace: Optional[torch.Tensor] = None):
    """Top-k pose retrieval. bank_c2w [N,4,4] f32, query_c2w [Q,4,4] f32,
    query_chunk [Q] i32. Returns (idx [Q,k] i32, score [Q,k] f32,
    count [Q] i32, frame_sel [Q,k*F] i32 or None)."""
    dev = query_c2w.device
    N, Q = bank_c2w.shape[0], query_c2w.shape[0]
    _need(bank_c2w, "bank_c2w", torch.float32, (N, 4, 4), dev)
    _need(query_c2w, "query_c2w", torch.float32, (Q, 4, 4), dev)
    _need(query_chunk, "query_chunk", torch.int32, (Q,), dev)
    if out is None:
        idx = torch.empty((Q, k), dtype=torch.int32, device=dev)
        score = torch.empty((Q, k), dtype=torch.float32, device=dev)
        count = torch.empty((Q,), dtype=torch.int32, device=dev)
        sel = (torch.empty((Q, k * frames_per_chunk), dtype=torch.int32, device=dev)
               if frames_per_chunk is not None else None)
    else:
        idx, score, count, sel = out
        _need(idx, "out idx", torch.int32, (Q, k), dev)
        _need(score, "out score", torch.float32, (Q, k), dev)
        _need(count, "out count", torch.int32, (Q,), dev)
        if (sel is None) != (frames_per_chunk is None):
            raise ValueError("out frame_sel must be given exactly when frames_per_chunk is")
        if sel is not None:
            _need(sel, "out frame_sel", torch.int32, (Q, k * frames_per_chunk), dev)
    ws = _workspace(retrieve_workspace_size(N, Q, k), workspace, dev, "workspace")
    st = lib().retrieve_chunks(_ptr(bank_c2w), N, _ptr(query_c2w), _ptr(query_chunk), Q, E, w_v, tau_c, tau_v,
                               delta, first_candidate, k, _ptr(idx), _ptr(score), _ptr(count),
                               frames_per_chunk or 0, _ptr(sel), _ptr(ws), ws.numel() if ws is not None else 0,
                               _stream(dev))
    _lib.check("retrieve_chunks", st)
    return idx, score, count, sel


def reproject_correspondence(tgt_depth: torch.Tensor, tgt_c2w: torch.Tensor, tgt_K: torch.Tensor,
                             src_depth: torch.Tensor, src_c2w: torch.Tensor, src_K: torch.Tensor, *,
                             p: int, eps: float, src_sel: Optional[torch.Tensor] = None, out=None):
    """Correspondence of every target token into every source frame.

    Batched: tgt_depth [B,Tq,h*p,w*p], tgt_c2w [B,Tq,4,4], tgt_K [B,Tq,4];
    sources [B,S,...] or, with src_sel [B,S] i32, a frame bank [n_src,...].
    Unbatched inputs (no leading B) give unbatched outputs.
    Returns (uv [B,S,Tq*h*w,2] f32, idx [B,S,Tq*h*w] i32)."""
    batched = tgt_depth.dim() == 4
    if not batched:
        tgt_depth, tgt_c2w, tgt_K = tgt_depth[None], tgt_c2w[None], tgt_K[None]
        if src_sel is None:
            src_depth, src_c2w, src_K = src_depth[None], src_c2w[None], src_K[None]
        else:
            src_sel = src_sel[None]
    dev = tgt_depth.device
    B, Tq, Hd, Wd = tgt_depth.shape
    if Hd % p or Wd % p:
        raise ValueError(f"depth map {Hd}x{Wd} is not a whole number of {p}x{p} tokens")
    h, w = Hd // p, Wd // p
    _need(tgt_depth, "tgt_depth", torch.float32, None, dev)
    _need(tgt_c2w, "tgt_c2w", torch.float32, (B, Tq, 4, 4), dev)
    _need(tgt_K, "tgt_K", torch.float32, (B, Tq, 4), dev)
    if src_sel is None:
        S = src_depth.shape[1]
        _need(src_depth, "src_depth", torch.float32, (B, S, Hd, Wd), dev)
        _need(src_c2w, "src_c2w", torch.float32, (B, S, 4, 4), dev)
        _need(src_K, "src_K", torch.float32, (B, S, 4), dev)
        n_src = 0
    else:
        S = src_sel.shape[1]
        n_src = src_depth.shape[0]
        _need(src_sel, "src_sel", torch.int32, (B, S), dev)
        _need(src_depth, "src_depth", torch.float32, (n_src, Hd, Wd), dev)
        _need(src_c2w, "src_c2w", torch.float32, (n_src, 4, 4), dev)
        _need(src_K, "src_K", torch.float32, (n_src, 4), dev)
    Lq = Tq * h * w
    if out is None:
        uv = torch.empty((B, S, Lq, 2), dtype=torch.float32, device=dev)
        idx = torch.empty((B, S, Lq), dtype=torch.int32, device=dev)
    else:
        uv, idx = out
        _need(uv, "out uv", torch.float32, (B, S, Lq, 2), dev)
        _need(idx, "out idx", torch.int32, (B, S, Lq), dev)
    st = lib().reproject_correspondence(_ptr(tgt_depth), _ptr(tgt_c2w), _ptr(tgt_K), _ptr(src_depth),
                                        _ptr(src_c2w), _ptr(src_K), _ptr(src_sel), n_src, B, Tq, S, h, w, p,
                                        eps, _ptr(uv), _ptr(idx), _stream(dev))
    _lib.check("reproject_correspondence", st)
    if not batched:
        return uv[0], idx[0]
    return uv, idx


def reproject_rotation(tgt_c2w: torch.Tensor, tgt_K: torch.Tensor, src_c2w: torch.Tensor, src_K: torch.Tensor, *,
                       h: int, w: int, p: int, src_sel: Optional[torch.Tensor] = None, out=None):
    """Rotation-only correspondence (sources sharing the target's centre): the
    homography u^ = pi(K_s R_s^T R_t K_t^-1 u~), no depth, no visibility test.

    Batched: tgt_c2w [B,Tq,4,4], tgt_K [B,Tq,4]; sources [B,S,...] or, with
    src_sel [B,S] i32, a frame bank [n_src,...]; h, w the token grid, p the
    latent pixels per token side (K is in depth-map pixels). Unbatched inputs
    give unbatched outputs. Returns (uv [B,S,Tq*h*w,2] f32, idx [B,S,Tq*h*w]
    i32), idx = REVISIT_CENTRE_MOVED (-6) for a pair whose centres differ."""
    batched = tgt_c2w.dim() == 4
    if not batched:
        tgt_c2w, tgt_K = tgt_c2w[None], tgt_K[None]
        if src_sel is None:
            src_c2w, src_K = src_c2w[None], src_K[None]
        else:
            src_sel = src_sel[None]
    dev = tgt_c2w.device
    if tgt_c2w.dim() != 4:
        raise ValueError(f"tgt_c2w must be [B,Tq,4,4] or [Tq,4,4] (got {tuple(tgt_c2w.shape)})")
    B, Tq = tgt_c2w.shape[:2]
    _need(tgt_c2w, "tgt_c2w", torch.float32, (B, Tq, 4, 4), dev)
    _need(tgt_K, "tgt_K", torch.float32, (B, Tq, 4), dev)
    if src_sel is None:
        S = src_c2w.shape[1]
        _need(src_c2w, "src_c2w", torch.float32, (B, S, 4, 4), dev)
        _need(src_K, "src_K", torch.float32, (B, S, 4), dev)
        n_src = 0
    else:
        S = src_sel.shape[1]
        n_src = src_c2w.shape[0]
        _need(src_sel, "src_sel", torch.int32, (B, S), dev)
        _need(src_c2w, "src_c2w", torch.float32, (n_src, 4, 4), dev)
        _need(src_K, "src_K", torch.float32, (n_src, 4), dev)
    Lq = Tq * h * w
    if out is None:
        uv = torch.empty((B, S, Lq, 2), dtype=torch.float32, device=dev)
        idx = torch.empty((B, S, Lq), dtype=torch.int32, device=dev)
    else:
        uv, idx = out
        _need(uv, "out uv", torch.float32, (B, S, Lq, 2), dev)
        _need(idx, "out idx", torch.int32, (B, S, Lq), dev)
    st = lib().reproject_rotation(_ptr(tgt_c2w), _ptr(tgt_K), _ptr(src_c2w), _ptr(src_K), _ptr(src_sel), n_src,
                                  B, Tq, S, h, w, p, _ptr(uv), _ptr(idx), _stream(dev))
    _lib.check("reproject_rotation", st)
    if not batched:
        return uv[0], idx[0]
    return uv, idx


def biased_chunk_attention(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, kv_frame_slot: torch.Tensor,
                           corr_uv: Optional[torch.Tensor], corr_idx: Optional[torch.Tensor], *,
                           h: int, w: int, softmax_scale: float, lam: float, sigma: float,
                           return_lse: bool = True, out=None, key_parts: int = 0,
                           workspace: Optional[torch.Tensor] = None, noalloc: bool = False):
    """Attention with the Gaussian correspondence bias on retrieved-frame keys.

    q [Lq,H,D], k, v [Lk,H,D] (bf16 with D=128, or fp32 with D in {64,128}, or
    q, k float8_e4m3fn with v bf16 and D=128: fp8 logits, o bf16);
    kv_frame_slot [Lk/(h*w)] i32; corr_uv [S,Lq,2] f32 and corr_idx [S,Lq] i32
    (None = no bias). key_parts: 0 = automatic key split, else a fixed
    number of parts (1..64). noalloc=True calls
    biased_chunk_attention_noalloc (the library's per-device scratch array
    instead of a workspace; with out= given nothing is allocated). Returns
    (o [Lq,H,D], lse [H,Lq] f32 or None)."""
    dev = q.device
    Lq, H, D = q.shape
    Lk = k.shape[0]
    dt = _attn_dtype(q.dtype)
    vdt = torch.bfloat16 if dt == FP8_QK else q.dtype  # fp8 q, k come with bf16 v, o
    _need(q, "q", q.dtype, None, dev)
    _need(k, "k", q.dtype, (Lk, H, D), dev)
    _need(v, "v", vdt, (Lk, H, D), dev)
    if Lk % (h * w):
        raise ValueError(f"Lk={Lk} is not a whole number of {h}x{w} frames")
    _need(kv_frame_slot, "kv_frame_slot", torch.int32, (Lk // (h * w),), dev)
    S = 0
    if corr_uv is not None:
        S = corr_uv.shape[0]
        _need(corr_uv, "corr_uv", torch.float32, (S, Lq, 2), dev)
        _need(corr_idx, "corr_idx", torch.int32, (S, Lq), dev)
    if out is None:
        o = torch.empty((Lq, H, D), dtype=vdt, device=dev)
        lse = torch.empty((H, Lq), dtype=torch.float32, device=dev) if return_lse else None
    else:
        o, lse = out
        _need(o, "o", vdt, (Lq, H, D), dev)
        if lse is not None:
            _need(lse, "lse", torch.float32, (H, Lq), dev)
    if noalloc:
        if workspace is not None:
            raise ValueError("noalloc=True takes no workspace (it uses the library's scratch array)")
        st = lib().biased_chunk_attention_noalloc(_ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(lse), dt, Lq, Lk, H, D, h,
                                                  w, _ptr(kv_frame_slot), _ptr(corr_uv), _ptr(corr_idx), S,
                                                  softmax_scale, lam, sigma, int(key_parts), _stream(dev))
        _lib.check("biased_chunk_attention_noalloc", st)
        return o, lse
    with torch.cuda.device(dev):
        nbytes = attention_workspace_size(q.dtype, Lq, Lk, H, D, key_parts)
    ws = _workspace(nbytes, workspace, dev, "workspace")
    st = lib().biased_chunk_attention(_ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(lse), dt, Lq, Lk, H, D, h, w,
                                      _ptr(kv_frame_slot), _ptr(corr_uv), _ptr(corr_idx), S,
                                      softmax_scale, lam, sigma, int(key_parts), _ptr(ws),
                                      ws.numel() if ws is not None else 0, _stream(dev))
    _lib.check("biased_chunk_attention", st)
    return o, lse


def pack_retrieved_kv(store_k: torch.Tensor, store_v: torch.Tensor, sel: torch.Tensor,
                      cache_k: torch.Tensor, cache_v: torch.Tensor, *, F: int, h: int, w: int,
                      dst_pos: int, dst_row0: int, rope_t_pairs: int, rope_theta: float,
                      store_pos: Optional[torch.Tensor] = None) -> None:
    """Copy the selected chunks' keys and values into the cache slots, in place.

    store_k, store_v [L, n_store, F*h*w, H, D]; cache_k, cache_v [L, rows, H, D]
    (bf16 or fp32, D a multiple of 8); sel [n_sel] i32 (entries outside
    [0, n_store) leave their slot untouched); store_pos None or [n_store] i32.
    Slot s goes to cache rows dst_row0 + s*F*h*w and frame position
    dst_pos + s*F; the first rope_t_pairs pairs of each key are re-rotated."""
    dev = cache_k.device
    if store_k.dim() != 5 or cache_k.dim() != 4:
        raise ValueError("store_k must be [L, n_store, T, H, D] and cache_k [L, rows, H, D]")
    L, n_store, T, H, D = store_k.shape
    rows = cache_k.shape[1]
    if cache_k.dtype == torch.bfloat16:
        dt = BF16
    elif cache_k.dtype == torch.float32:
        dt = F32
    else:
        raise TypeError(f"cache_k must be bfloat16 or float32 (got {cache_k.dtype})")
    if T != F * h * w:
        raise ValueError(f"store rows per chunk {T} != F*h*w = {F * h * w}")
    _need(store_k, "store_k", cache_k.dtype, (L, n_store, T, H, D), dev)
    _need(store_v, "store_v", cache_k.dtype, (L, n_store, T, H, D), dev)
    _need(cache_k, "cache_k", cache_k.dtype, (L, rows, H, D), dev)
    _need(cache_v, "cache_v", cache_k.dtype, (L, rows, H, D), dev)
    _need(sel, "sel", torch.int32, None, dev)
    if store_pos is not None:
        _need(store_pos, "store_pos", torch.int32, (n_store,), dev)
    st = lib().pack_retrieved_kv(_ptr(store_k), _ptr(store_v), _ptr(store_pos), n_store, _ptr(sel), sel.numel(),
                                 int(dst_pos), _ptr(cache_k), _ptr(cache_v), int(dst_row0), rows, L, dt, F, h, w, H,
                                 D, int(rope_t_pairs), float(rope_theta), _stream(dev))
    _lib.check("pack_retrieved_kv", st)


def pool_token_depth(depth: torch.Tensor, p: int, out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Token depth [n, h, w] f32 from depth maps [n, h*p, w*p] f32 (p x p means, fp32)."""
    dev = depth.device
    if depth.dim() != 3 or depth.shape[1] % p or depth.shape[2] % p:
        raise ValueError("depth must be [n, h*p, w*p]")
    n, Hd, Wd = depth.shape
    h, w = Hd // p, Wd // p
    _need(depth, "depth", torch.float32, (n, Hd, Wd), dev)
    if out is None:
        out = torch.empty((n, h, w), dtype=torch.float32, device=dev)
    _need(out, "out", torch.float32, (n, h, w), dev)
    _lib.check("pool_token_depth", lib().pool_token_depth(_ptr(depth), n, h, w, p, _ptr(out), _stream(dev)))
    return out


class StreamDriver:
    """The paper's cache layout run chunk by chunk on the device (rc_stream_*).

    Owns a stream object: history ring of ``capacity`` chunks, pose bank of
    ``max_chunks``, packed cache. ``step`` runs the next chunk: depth
    [F, h*p, w*p] f32, c2w [F, 4, 4] f32, K [F, 4] f32, q, k, v
    [layers, F*h*w, H, D] (bf16 or f32, k embedded at positions 4F + f);
    returns o [layers, F*h*w, H, D] and lse [layers, H, F*h*w]."""

    def __init__(self, *, F: int, h: int, w: int, p: int, H: int, D: int, layers: int, dtype: torch.dtype,
                 capacity: int, max_chunks: int, E: float, w_v: float, tau_c: float, tau_v: float, delta: int,
                 eps: float, lam: float, sigma: float, softmax_scale: float, rope_t_pairs: int, rope_theta: float):
        if dtype == torch.bfloat16:
            dt = BF16
        elif dtype == torch.float32:
            dt = F32
        else:
            raise TypeError(f"dtype must be bfloat16 or float32 (got {dtype})")
        self.dtype = dtype
        self.F, self.h, self.w, self.p, self.H, self.D, self.layers = F, h, w, p, H, D, layers
        cfg = _lib.StreamConfig(F=F, h=h, w=w, p=p, H=H, D=D, layers=layers, dtype=dt, capacity=capacity,
                                max_chunks=max_chunks, E=E, w_v=w_v, tau_c=tau_c, tau_v=tau_v, delta=delta, eps=eps,
                                lam=lam, sigma=sigma, softmax_scale=softmax_scale, rope_t_pairs=rope_t_pairs,
                                rope_theta=rope_theta)
        handle = ctypes.c_void_p(0)
        _lib.check("rc_stream_create", lib().rc_stream_create(ctypes.byref(cfg), ctypes.byref(handle)))
        self._h = handle

    def step(self, depth, c2w, K, q, k, v, out=None):
        if not self._h:
            raise RuntimeError("stream already closed")
        dev = q.device
        T = self.F * self.h * self.w
        _need(depth, "depth", torch.float32, (self.F, self.h * self.p, self.w * self.p), dev)
        _need(c2w, "c2w", torch.float32, (self.F, 4, 4), dev)
        _need(K, "K", torch.float32, (self.F, 4), dev)
        shape = (self.layers, T, self.H, self.D)
        for t, name in ((q, "q"), (k, "k"), (v, "v")):
            _need(t, name, self.dtype, shape, dev)
        if out is None:
            o = torch.empty(shape, dtype=self.dtype, device=dev)
            lse = torch.empty((self.layers, self.H, T), dtype=torch.float32, device=dev)
        else:
            o, lse = out
            _need(o, "o", self.dtype, shape, dev)
            if lse is not None:
                _need(lse, "lse", torch.float32, (self.layers, self.H, T), dev)
        st = lib().rc_stream_step(self._h, _ptr(depth), _ptr(c2w), _ptr(K), _ptr(q), _ptr(k), _ptr(v), _ptr(o),
                                  _ptr(lse), _stream(dev))
        _lib.check("rc_stream_step", st)
        return o, lse

    def state(self):
        """The last step's layout sizes and device pointers (rc_stream_state)."""
        stt = _lib.StreamState()
        _lib.check("rc_stream_view", lib().rc_stream_view(self._h, ctypes.byref(stt)))
        return stt

    def close(self):
        if self._h:
            lib().rc_stream_destroy(self._h)
            self._h = ctypes.c_void_p(0)

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
