"""ctypes loader for librevisit.so (the C interface in include/revisit.h).

The library is built in-tree by ``paper_2607_21848_amd.build``. There is no
fallback: if the shared library is missing or fails to load, every entry
point raises.
"""

from __future__ import annotations

import ctypes
import os

_LIB = None
LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "librevisit.so")

OK, ERR_NULL, ERR_SHAPE, ERR_UNSUPPORTED, ERR_PARAM, ERR_LAUNCH, ERR_MEMORY = 0, 1, 2, 3, 4, 5, 6
BF16, F32, FP8_QK = 1, 2, 3
MAX_K = 32
EXPORTED = ("rc_status_string", "rc_last_error", "retrieve_chunks", "reproject_correspondence",
            "reproject_rotation", "biased_chunk_attention", "biased_chunk_attention_noalloc", "rc_retrieve_workspace_size",
            "rc_attention_workspace_size",
            "pack_retrieved_kv", "pool_token_depth", "rc_stream_create", "rc_stream_step", "rc_stream_view",
            "rc_stream_destroy")

_p = ctypes.c_void_p
_i = ctypes.c_int32
_f = ctypes.c_float
_z = ctypes.c_size_t


class StreamConfig(ctypes.Structure):
    """rc_stream_config of include/revisit.h."""
    _fields_ = [(n, ctypes.c_int32) for n in ("F", "h", "w", "p", "H", "D", "layers", "dtype", "capacity",
                                               "max_chunks")] + \
               [(n, ctypes.c_float) for n in ("E", "w_v", "tau_c", "tau_v")] + [("delta", ctypes.c_int32)] + \
               [(n, ctypes.c_float) for n in ("eps", "lam", "sigma", "softmax_scale")] + \
               [("rope_t_pairs", ctypes.c_int32), ("rope_theta", ctypes.c_float)]


class StreamState(ctypes.Structure):
    """rc_stream_state of include/revisit.h."""
    _fields_ = [(n, ctypes.c_int32) for n in ("n", "n_parts", "ret_part", "Lk", "cache_rows")] + \
               [(n, ctypes.c_void_p) for n in ("ret_idx", "ret_count", "part_slot", "kv_slot", "src_sel", "corr_uv",
                                               "corr_idx", "cache_k", "cache_v")]


class RevisitError(RuntimeError):
    def __init__(self, fn: str, status: int, detail: str):
        super().__init__(f"{fn}: status {status} ({status_string(status)}): {detail}")
        self.status = status


def lib() -> ctypes.CDLL:
    """The loaded library (loaded once)."""
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"librevisit.so not found at {LIB_PATH}: build it with "
                               "`python -m paper_2607_21848_amd.build` (there is no CPU fallback)")
        L = ctypes.CDLL(LIB_PATH)
        L.rc_status_string.restype = ctypes.c_char_p
        L.rc_status_string.argtypes = [ctypes.c_int]
        L.rc_last_error.restype = ctypes.c_char_p
        L.rc_last_error.argtypes = []
        L.retrieve_chunks.restype = ctypes.c_int
        L.retrieve_chunks.argtypes = [_p, _i, _p, _p, _i, _f, _f, _f, _f, _i, _i, _i, _p, _p, _p, _i, _p, _p, _z,
                                      _p]
        L.rc_retrieve_workspace_size.restype = ctypes.c_int
        L.rc_retrieve_workspace_size.argtypes = [_i, _i, _i, ctypes.POINTER(ctypes.c_size_t)]
        L.reproject_correspondence.restype = ctypes.c_int
        L.reproject_correspondence.argtypes = [_p, _p, _p, _p, _p, _p, _p, _i, _i, _i, _i, _i, _i, _i, _f,
                                               _p, _p, _p]
        L.reproject_rotation.restype = ctypes.c_int
        L.reproject_rotation.argtypes = [_p, _p, _p, _p, _p, _i, _i, _i, _i, _i, _i, _i, _p, _p, _p]
        L.biased_chunk_attention.restype = ctypes.c_int
        L.biased_chunk_attention.argtypes = [_p, _p, _p, _p, _p, _i, _i, _i, _i, _i, _i, _i, _p, _p, _p, _i,
                                             _f, _f, _f, _i, _p, _z, _p]
        L.biased_chunk_attention_noalloc.restype = ctypes.c_int
        L.biased_chunk_attention_noalloc.argtypes = [_p, _p, _p, _p, _p, _i, _i, _i, _i, _i, _i, _i, _p, _p, _p, _i,
                                                     _f, _f, _f, _i, _p]
        L.rc_attention_workspace_size.restype = ctypes.c_int
        L.rc_attention_workspace_size.argtypes = [_i, _i, _i, _i, _i, _i, ctypes.POINTER(ctypes.c_size_t)]
        L.pack_retrieved_kv.restype = ctypes.c_int
        L.pack_retrieved_kv.argtypes = [_p, _p, _p, _i, _p, _i, _i, _p, _p, _i, _i, _i, _i, _i, _i, _i, _i, _i, _i,
                                        _f, _p]
        L.pool_token_depth.restype = ctypes.c_int
        L.pool_token_depth.argtypes = [_p, _i, _i, _i, _i, _p, _p]
        L.rc_stream_create.restype = ctypes.c_int
        L.rc_stream_create.argtypes = [ctypes.POINTER(StreamConfig), ctypes.POINTER(ctypes.c_void_p)]
        L.rc_stream_step.restype = ctypes.c_int
        L.rc_stream_step.argtypes = [_p, _p, _p, _p, _p, _p, _p, _p, _p, _p]
        L.rc_stream_view.restype = ctypes.c_int
        L.rc_stream_view.argtypes = [_p, ctypes.POINTER(StreamState)]
        L.rc_stream_destroy.restype = ctypes.c_int
        L.rc_stream_destroy.argtypes = [_p]
        _LIB = L
    return _LIB


def status_string(status: int) -> str:
    return lib().rc_status_string(int(status)).decode()


def last_error() -> str:
    return lib().rc_last_error().decode()


def check(fn: str, status: int) -> None:
    if status != OK:
        raise RevisitError(fn, status, last_error())
