"""ctypes view of libwushkv.so (include/wushkv.h).

Argument marshalling only: every step of the hot path runs in the HIP
kernels behind these entry points.  There is no CPU fallback; if the
library is missing, loading fails loudly.
"""
from __future__ import annotations

import ctypes
import os
import re

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "_build", "libwushkv.so")
HEADER = os.path.join(os.path.dirname(_HERE), "include", "wushkv.h")

OK, EINVAL, EUNSUPPORTED, EWORKSPACE, ELAUNCH, ENODEVICE = 0, -1, -2, -3, -4, -5
NOALLOC_SCRATCH_BYTES = 32 << 20  # WUSHKV_NOALLOC_SCRATCH_BYTES
CODEC_PCLIP, CODEC_QUEST = 0, 1
PAGE_TOKENS = 64


class CacheDesc(ctypes.Structure):
    """Mirror of struct wushkv_cache."""
    _fields_ = [
        ("batch", ctypes.c_int32),
        ("n_kv_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("bits", ctypes.c_int32),
        ("s_sink", ctypes.c_int32),
        ("s_keep", ctypes.c_int32),
        ("s_flush", ctypes.c_int32),
        ("win_slots", ctypes.c_int32),
        ("max_pages_per_seq", ctypes.c_int32),
        ("n_pages", ctypes.c_int32),
        ("kappa_k", ctypes.c_float),
        ("kappa_v", ctypes.c_float),
        ("codec", ctypes.c_int32),
        ("quest_alpha", ctypes.c_float),
        ("pages", ctypes.c_void_p),
        ("page_table", ctypes.c_void_p),
        ("win_k", ctypes.c_void_p),
        ("win_v", ctypes.c_void_p),
        ("seq_len", ctypes.c_void_p),
        ("quant_end", ctypes.c_void_p),
        ("commit", ctypes.c_void_p),
    ]


class WushKVError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__("%s failed: %s (%d)" % (where, status_string(status), status))


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(
                "libwushkv.so is not built (%s); run `python -m paper_2609_38121_amd.build`"
                % LIB_PATH)
        L = ctypes.CDLL(LIB_PATH)
        _declare(L)
        _lib = L
    return _lib


def _declare(L):
    P, I32, F32, SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_float, ctypes.c_size_t
    D = ctypes.POINTER(CacheDesc)
    L.wushkv_page_bytes.argtypes = [I32, I32]
    L.wushkv_page_bytes.restype = SZ
    L.wushkv_append.argtypes = [D, P, P, P, I32, P, P, P]
    L.wushkv_append.restype = ctypes.c_int
    L.wushkv_append_norm_rope.argtypes = [D, P, P, P, I32, P, P, F32, P, I32, P, P]
    L.wushkv_append_norm_rope.restype = ctypes.c_int
    L.wushkv_decode_attention.argtypes = [D, P, I32, I32, P, F32, P, P, SZ, P]
    L.wushkv_decode_attention.restype = ctypes.c_int
    L.wushkv_decode_attention_noalloc.argtypes = [D, P, I32, I32, P, F32, P, P]
    L.wushkv_decode_attention_noalloc.restype = ctypes.c_int
    L.wushkv_decode_workspace_bytes.argtypes = [D, I32, I32]
    L.wushkv_decode_workspace_bytes.restype = SZ
    L.wushkv_decode_step.argtypes = [D, P, P, P, P, P, I32, I32, P, F32, P, P, SZ, P]
    L.wushkv_decode_step.restype = ctypes.c_int
    L.wushkv_chunk_attention.argtypes = [D, P, P, I32, I32, I32, P, F32, P, P, SZ, P]
    L.wushkv_chunk_attention.restype = ctypes.c_int
    L.wushkv_chunk_workspace_bytes.argtypes = [D, I32, I32, I32]
    L.wushkv_chunk_workspace_bytes.restype = SZ
    L.wushkv_dequant.argtypes = [D, I32, I32, I32, P, P, P]
    L.wushkv_dequant.restype = ctypes.c_int
    L.wushkv_status_string.argtypes = [ctypes.c_int]
    L.wushkv_status_string.restype = ctypes.c_char_p
    L.wushkv_abi_version.argtypes = []
    L.wushkv_abi_version.restype = ctypes.c_int
    L.wushkv_wush_transform.argtypes = [P, P, I32, I32, F32, P, P, P, P]
    L.wushkv_wush_transform.restype = ctypes.c_int
    L.wushkv_read_probe.argtypes = [P, SZ, I32, P, P]
    L.wushkv_read_probe.restype = ctypes.c_int
    L.wushkv_quest_alpha.argtypes = [I32]
    L.wushkv_quest_alpha.restype = ctypes.c_double
    L.wushkv_timing_enable.argtypes = [I32]
    L.wushkv_timing_enable.restype = ctypes.c_int
    L.wushkv_timing_read.argtypes = [ctypes.c_char_p, ctypes.POINTER(I32),
                                     ctypes.POINTER(ctypes.c_double)]
    L.wushkv_timing_read.restype = ctypes.c_int
    L.wushkv_timing_count.argtypes = []
    L.wushkv_timing_count.restype = ctypes.c_int
    L.wushkv_timing_launch.argtypes = [I32, ctypes.POINTER(ctypes.c_char_p),
                                       ctypes.POINTER(ctypes.c_double)]
    L.wushkv_timing_launch.restype = ctypes.c_int


def header_functions() -> list[str]:
    """Names of the functions include/wushkv.h declares."""
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[\w\s\*]+?\b(wushkv_\w+)\s*\(", text, re.M)))


def status_string(status: int) -> str:
    return lib().wushkv_status_string(status).decode()


def check(status: int, where: str) -> None:
    if status != OK:
        raise WushKVError(status, where)
