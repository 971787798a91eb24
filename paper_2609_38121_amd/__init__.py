"""WUSH-KV online hot path for AMD Instinct MI355X (gfx950).

Python binding over the C ABI in include/wushkv.h.  The functions here have
the names of the C entry points and only marshal arguments; PyTorch supplies
device memory and the current HIP stream.

    cache = WushKVCache(batch=8, n_kv_heads=8, head_dim=128, bits=2,
                        s_sink=4, s_keep=128, s_flush=8,
                        kappa_k=0.96, kappa_v=0.92, max_seq_len=8192)
    wushkv_append(cache, k_new, v_new, n_new, t_k)
    out = wushkv_decode_attention(cache, q, t_k_inv)
"""
from __future__ import annotations

import ctypes
import math

from . import _lib
from ._lib import (CacheDesc, WushKVError, PAGE_TOKENS, check, header_functions,
                   status_string)

__all__ = [
    "WushKVCache", "WushKVError", "wushkv_append", "wushkv_decode_attention",
    "wushkv_decode_attention_noalloc", "wushkv_decode_step",
    "wushkv_decode_workspace_bytes", "wushkv_dequant", "wushkv_page_bytes",
    "wushkv_status_string", "wushkv_abi_version", "wushkv_timing_enable",
    "wushkv_timing_read", "wushkv_timing_launches", "wushkv_quest_alpha", "wushkv_wush_transform", "wushkv_read_probe",
    "PAGE_TOKENS",
    "header_functions",
]


def _torch():
    import torch
    return torch


def _ptr(t) -> int | None:
    return None if t is None else t.data_ptr()


def _stream_handle(stream) -> int:
    torch = _torch()
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


def wushkv_page_bytes(head_dim: int, bits: int) -> int:
    return _lib.lib().wushkv_page_bytes(head_dim, bits)


def wushkv_status_string(status: int) -> str:
    return status_string(status)


def wushkv_abi_version() -> int:
    return _lib.lib().wushkv_abi_version()


def wushkv_quest_alpha(bits: int) -> float:
    """The Gaussian-MSE-optimal clip multiplier alpha_b of Eq. (5)."""
    return _lib.lib().wushkv_quest_alpha(bits)


def wushkv_timing_enable(slots: int) -> None:
    check(_lib.lib().wushkv_timing_enable(slots), "wushkv_timing_enable")


def wushkv_timing_read(name_substr: str = ""):
    """(launch count, summed milliseconds per launch) of recorded launches
    whose kernel name contains name_substr; reading does not clear the
    record (re-enabling does)."""
    cnt = ctypes.c_int32()
    ms = ctypes.c_double()
    check(_lib.lib().wushkv_timing_read(name_substr.encode(), ctypes.byref(cnt),
                                        ctypes.byref(ms)), "wushkv_timing_read")
    return cnt.value, ms.value


def wushkv_timing_launches():
    """[(kernel name, milliseconds)] of every launch recorded since timing
    was enabled, in launch order."""
    L = _lib.lib()
    out = []
    name = ctypes.c_char_p()
    ms = ctypes.c_double()
    for i in range(L.wushkv_timing_count()):
        check(L.wushkv_timing_launch(i, ctypes.byref(name), ctypes.byref(ms)), "wushkv_timing_launch")
        out.append((name.value.decode(), ms.value))
    return out


class WushKVCache:
    """Device memory of one WUSH-KV cache plus its C descriptor.

    Allocates (torch, on ``device``): the page pool, the page table, the bf16
    windows, the per-sequence counters and the append's arrival counts, all
    zero-initialised except the windows, which may hold anything (they are
    only read where live).
    ``page_order`` "linear" maps logical page i of sequence b to physical
    page b * max_pages + i; "random" draws a seeded permutation of a pool
    ``pool_factor`` times the needed size.  ``codec`` is "pclip" (Eq. (7),
    clip quantiles kappa_k / kappa_v) or "quest" (Eq. (5), clip multiplier
    ``quest_alpha``, by default the library's wushkv_quest_alpha(bits)).
    """

    def __init__(self, batch, n_kv_heads, head_dim, bits, s_sink, s_keep, s_flush,
                 kappa_k, kappa_v, max_seq_len, win_slots=None, page_order="linear",
                 pool_factor=1.0, seed=0, device="cuda", codec="pclip", quest_alpha=None):
        torch = _torch()
        self.batch, self.n_kv_heads, self.head_dim, self.bits = batch, n_kv_heads, head_dim, bits
        self.s_sink, self.s_keep, self.s_flush = s_sink, s_keep, s_flush
        self.kappa_k, self.kappa_v = float(kappa_k), float(kappa_v)
        codes = {"pclip": _lib.CODEC_PCLIP, "quest": _lib.CODEC_QUEST}
        if codec not in codes:
            raise ValueError(codec)
        self.codec = codec
        if quest_alpha is None:
            quest_alpha = wushkv_quest_alpha(bits) if codec == "quest" else 0.0
        self.quest_alpha = float(ctypes.c_float(quest_alpha).value)  # as the descriptor holds it
        self.max_seq_len = max_seq_len
        if win_slots is None:
            need = s_sink + max(1, s_keep + s_flush - 1)
            win_slots = PAGE_TOKENS * math.ceil(need / PAGE_TOKENS)
        self.win_slots = win_slots
        self.max_pages = max(1, math.ceil(max(0, max_seq_len - s_sink) / PAGE_TOKENS))
        need_pages = batch * self.max_pages
        self.n_pages = max(need_pages, int(math.ceil(need_pages * pool_factor)))
        self.page_bytes = wushkv_page_bytes(head_dim, bits)
        if self.page_bytes == 0:
            raise WushKVError(_lib.EUNSUPPORTED, "WushKVCache")
        dev = torch.device(device)
        self.device = dev
        self.pages = torch.zeros(self.n_pages * n_kv_heads * self.page_bytes, dtype=torch.uint8,
                                 device=dev)
        if page_order == "linear":
            table = torch.arange(need_pages, dtype=torch.int32)
        elif page_order == "random":
            g = torch.Generator().manual_seed(seed)
            table = torch.randperm(self.n_pages, generator=g)[:need_pages].to(torch.int32)
        else:
            raise ValueError(page_order)
        self.page_table = table.reshape(batch, self.max_pages).contiguous().to(dev)
        self.win_k = torch.zeros(batch, n_kv_heads, win_slots, head_dim, dtype=torch.bfloat16,
                                 device=dev)
        self.win_v = torch.zeros(batch, n_kv_heads, head_dim, win_slots, dtype=torch.bfloat16,
                                 device=dev)
        self.seq_len = torch.zeros(batch, dtype=torch.int32, device=dev)
        self.quant_end = torch.zeros(batch, dtype=torch.int32, device=dev)
        self.commit = torch.zeros(batch, dtype=torch.int32, device=dev)
        self._desc = self._make_desc()

    def _make_desc(self) -> CacheDesc:
        return CacheDesc(
            self.batch, self.n_kv_heads, self.head_dim, self.bits, self.s_sink, self.s_keep,
            self.s_flush, self.win_slots, self.max_pages, self.n_pages, self.kappa_k,
            self.kappa_v, {"pclip": _lib.CODEC_PCLIP, "quest": _lib.CODEC_QUEST}[self.codec],
            self.quest_alpha, self.pages.data_ptr(), self.page_table.data_ptr(),
            self.win_k.data_ptr(), self.win_v.data_ptr(), self.seq_len.data_ptr(),
            self.quant_end.data_ptr(), self.commit.data_ptr())

    @property
    def desc(self) -> CacheDesc:
        return self._desc

    def clone(self) -> "WushKVCache":
        """Deep copy (same layout, same page table, fresh device memory)."""
        new = object.__new__(WushKVCache)
        new.__dict__.update({k: v for k, v in self.__dict__.items() if k != "_desc"})
        for name in ("pages", "page_table", "win_k", "win_v", "seq_len", "quant_end", "commit"):
            setattr(new, name, getattr(self, name).clone())
        new._desc = new._make_desc()
        return new


def _check_2byte(t, name):
    if t is None:
        return
    if t.element_size() != 2 or not t.is_contiguous():
        raise ValueError("%s must be a contiguous 2-byte (bf16) tensor" % name)


def wushkv_append(cache: WushKVCache, k_new, v_new, n_new, t_k, k_tilde_out=None,
                  max_new=None, stream=None) -> None:
    """Alg. 2 steps 3-4 and 7-11 on the GPU.  k_new / v_new: bf16
    [batch][max_new][n_kv][d]; n_new: int32 [batch] on the device; t_k: bf16
    [n_kv][d][d]."""
    for t, nm in ((k_new, "k_new"), (v_new, "v_new"), (t_k, "t_k"), (k_tilde_out, "k_tilde_out")):
        _check_2byte(t, nm)
    if max_new is None:
        max_new = k_new.shape[1]
    st = _lib.lib().wushkv_append(ctypes.byref(cache.desc), _ptr(k_new), _ptr(v_new),
                                  _ptr(n_new), int(max_new), _ptr(t_k), _ptr(k_tilde_out),
                                  _stream_handle(stream))
    check(st, "wushkv_append")


def wushkv_append_norm_rope(cache: WushKVCache, k_raw, v_new, n_new, t_k, rope_table,
                            norm_gain=None, norm_eps=0.0, k_tilde_out=None, max_new=None,
                            stream=None) -> None:
    """wushkv_append with the headwise RMS normalisation and the rotary
    embedding of the new keys fused in front (Alg. 2 step 1).  k_raw: bf16
    [batch][max_new][n_kv][d] projected keys; rope_table: fp32 [positions][d]
    (cos | sin); norm_gain: fp32 [d] or None."""
    for t, nm in ((k_raw, "k_raw"), (v_new, "v_new"), (t_k, "t_k"), (k_tilde_out, "k_tilde_out")):
        _check_2byte(t, nm)
    if rope_table.element_size() != 4 or not rope_table.is_contiguous():
        raise ValueError("rope_table must be a contiguous fp32 tensor")
    if max_new is None:
        max_new = k_raw.shape[1]
    st = _lib.lib().wushkv_append_norm_rope(
        ctypes.byref(cache.desc), _ptr(k_raw), _ptr(v_new), _ptr(n_new), int(max_new), _ptr(t_k),
        _ptr(norm_gain), float(norm_eps), _ptr(rope_table), int(rope_table.shape[0]),
        _ptr(k_tilde_out), _stream_handle(stream))
    check(st, "wushkv_append_norm_rope")


def wushkv_decode_workspace_bytes(cache: WushKVCache, n_q_heads: int, max_seq_len: int) -> int:
    return _lib.lib().wushkv_decode_workspace_bytes(ctypes.byref(cache.desc), n_q_heads,
                                                    max_seq_len)


def wushkv_decode_attention(cache: WushKVCache, q, t_k_inv, sm_scale=None, max_seq_len=None,
                            out=None, workspace=None, stream=None):
    """One decode query per query head.  q: bf16 [batch][n_q][d];
    t_k_inv: fp32 [n_kv][d][d].  Returns fp32 [batch][n_q][d]."""
    torch = _torch()
    _check_2byte(q, "q")
    n_q = q.shape[1]
    if max_seq_len is None:
        max_seq_len = cache.max_seq_len
    if sm_scale is None:
        sm_scale = 1.0 / math.sqrt(cache.head_dim)
    if out is None:
        out = torch.empty(cache.batch, n_q, cache.head_dim, dtype=torch.float32, device=q.device)
    need = wushkv_decode_workspace_bytes(cache, n_q, max_seq_len)
    if need == 0:
        raise WushKVError(_lib.EINVAL, "wushkv_decode_workspace_bytes")
    if workspace is None:
        workspace = torch.empty(need, dtype=torch.uint8, device=q.device)
    st = _lib.lib().wushkv_decode_attention(
        ctypes.byref(cache.desc), _ptr(q), n_q, int(max_seq_len), _ptr(t_k_inv),
        float(sm_scale), _ptr(out), _ptr(workspace), workspace.numel() * workspace.element_size(),
        _stream_handle(stream))
    check(st, "wushkv_decode_attention")
    return out


def wushkv_decode_attention_noalloc(cache: WushKVCache, q, t_k_inv, out, sm_scale=None,
                                    max_seq_len=None, stream=None):
    """wushkv_decode_attention with the library's static workspace: nothing
    is allocated (``out`` is the caller's fp32 [batch][n_q][d]).  Calls that
    overlap on one GPU race on that workspace."""
    _check_2byte(q, "q")
    n_q = q.shape[1]
    if max_seq_len is None:
        max_seq_len = cache.max_seq_len
    if sm_scale is None:
        sm_scale = 1.0 / math.sqrt(cache.head_dim)
    st = _lib.lib().wushkv_decode_attention_noalloc(
        ctypes.byref(cache.desc), _ptr(q), n_q, int(max_seq_len), _ptr(t_k_inv),
        float(sm_scale), _ptr(out), _stream_handle(stream))
    check(st, "wushkv_decode_attention_noalloc")
    return out


def wushkv_decode_step(cache: WushKVCache, k_new, v_new, n_new, t_k, q, t_k_inv, sm_scale=None,
                       max_seq_len=None, out=None, workspace=None, stream=None):
    """One decode step in Alg. 2's order: each sequence's new token (n_new[b]
    of 0 or 1) is appended, attention runs over the cache with it (the
    positions due for quantisation still at bf16), then the flush.
    k_new, v_new: bf16 [batch][n_kv][d]; n_new: int32 [batch] on the device;
    t_k: bf16 [n_kv][d][d]; q: bf16 [batch][n_q][d]; t_k_inv: fp32
    [n_kv][d][d].  Returns fp32 [batch][n_q][d]."""
    torch = _torch()
    _check_2byte(q, "q")
    _check_2byte(k_new, "k_new")
    _check_2byte(v_new, "v_new")
    _check_2byte(t_k, "t_k")
    n_q = q.shape[1]
    if max_seq_len is None:
        max_seq_len = cache.max_seq_len
    if sm_scale is None:
        sm_scale = 1.0 / math.sqrt(cache.head_dim)
    if out is None:
        out = torch.empty(cache.batch, n_q, cache.head_dim, dtype=torch.float32, device=q.device)
    need = wushkv_decode_workspace_bytes(cache, n_q, max_seq_len)
    if need == 0:
        raise WushKVError(_lib.EINVAL, "wushkv_decode_workspace_bytes")
    if workspace is None:
        workspace = torch.empty(need, dtype=torch.uint8, device=q.device)
    st = _lib.lib().wushkv_decode_step(
        ctypes.byref(cache.desc), _ptr(k_new), _ptr(v_new), _ptr(n_new), _ptr(t_k), _ptr(q), n_q,
        int(max_seq_len), _ptr(t_k_inv), float(sm_scale), _ptr(out), _ptr(workspace),
        workspace.numel() * workspace.element_size(), _stream_handle(stream))
    check(st, "wushkv_decode_step")
    return out


def wushkv_chunk_workspace_bytes(cache: WushKVCache, n_q_heads: int, max_tok: int,
                                 max_seq_len: int) -> int:
    return _lib.lib().wushkv_chunk_workspace_bytes(ctypes.byref(cache.desc), n_q_heads, max_tok,
                                                   max_seq_len)


def wushkv_chunk_attention(cache: WushKVCache, q, t_k_inv, n_tok=None, sm_scale=None,
                           max_seq_len=None, out=None, workspace=None, stream=None):
    """Attention of each sequence's chunk of new tokens, causal inside the
    chunk.  q: bf16 [batch][max_tok][n_q][d]; n_tok: int32 [batch] on the
    device or None (max_tok for all).  Returns fp32 [batch][max_tok][n_q][d]."""
    torch = _torch()
    _check_2byte(q, "q")
    max_tok, n_q = q.shape[1], q.shape[2]
    if max_seq_len is None:
        max_seq_len = cache.max_seq_len
    if sm_scale is None:
        sm_scale = 1.0 / math.sqrt(cache.head_dim)
    if out is None:
        out = torch.empty(cache.batch, max_tok, n_q, cache.head_dim, dtype=torch.float32,
                          device=q.device)
    need = wushkv_chunk_workspace_bytes(cache, n_q, max_tok, max_seq_len)
    if need == 0:
        raise WushKVError(_lib.EINVAL, "wushkv_chunk_workspace_bytes")
    if workspace is None:
        workspace = torch.empty(need, dtype=torch.uint8, device=q.device)
    st = _lib.lib().wushkv_chunk_attention(
        ctypes.byref(cache.desc), _ptr(q), _ptr(n_tok), int(max_tok), n_q, int(max_seq_len),
        _ptr(t_k_inv), float(sm_scale), _ptr(out), _ptr(workspace),
        workspace.numel() * workspace.element_size(), _stream_handle(stream))
    check(st, "wushkv_chunk_attention")
    return out


def wushkv_dequant(cache: WushKVCache, b: int, start: int, count: int, k_out=None, v_out=None,
                   stream=None):
    """fp32 [n_kv][count][d] reconstructions of stored positions
    [start, start + count) of sequence b.  Returns (k_out, v_out)."""
    torch = _torch()
    shape = (cache.n_kv_heads, count, cache.head_dim)
    if k_out is None:
        k_out = torch.empty(shape, dtype=torch.float32, device=cache.device)
    if v_out is None:
        v_out = torch.empty(shape, dtype=torch.float32, device=cache.device)
    st = _lib.lib().wushkv_dequant(ctypes.byref(cache.desc), int(b), int(start), int(count),
                                   _ptr(k_out), _ptr(v_out), _stream_handle(stream))
    check(st, "wushkv_dequant")
    return k_out, v_out


def wushkv_wush_transform(m, h, gamma: float = 1e-2, t_out=None, t_inv_out=None,
                          want_inverse: bool = True, sweeps_out=None, stream=None):
    """T = Wush(M, H, gamma) of Eq. (1) for each of the [count][d][d] fp32
    (device, symmetric) pairs in m and h.  Returns (T, T^{-1} or None,
    sweeps int32 [count]: Jacobi sweeps taken, -1 where a damped matrix was
    not positive definite)."""
    torch = _torch()
    if m.shape != h.shape or m.dim() != 3 or m.shape[1] != m.shape[2]:
        raise ValueError("m and h must both be [count][d][d]")
    count, d = int(m.shape[0]), int(m.shape[1])
    for t in (m, h):
        if t.dtype != torch.float32 or not t.is_contiguous():
            raise ValueError("m and h must be contiguous fp32")
    if t_out is None:
        t_out = torch.empty_like(m)
    if want_inverse and t_inv_out is None:
        t_inv_out = torch.empty_like(m)
    if sweeps_out is None:
        sweeps_out = torch.empty(count, dtype=torch.int32, device=m.device)
    st = _lib.lib().wushkv_wush_transform(_ptr(m), _ptr(h), count, d, float(gamma), _ptr(t_out),
                                          _ptr(t_inv_out) if want_inverse else None,
                                          _ptr(sweeps_out), _stream_handle(stream))
    check(st, "wushkv_wush_transform")
    return t_out, (t_inv_out if want_inverse else None), sweeps_out


def wushkv_read_probe(buf, mode: int, sink=None, stream=None):
    """Streaming read of the device tensor buf (byte size a multiple of
    65536), mode 0 vector loads or 1 direct-to-LDS loads.  Returns sink."""
    torch = _torch()
    nbytes = buf.numel() * buf.element_size()
    if sink is None:
        sink = torch.empty(max(1, nbytes // 65536), dtype=torch.int32, device=buf.device)
    check(_lib.lib().wushkv_read_probe(_ptr(buf), nbytes, int(mode), _ptr(sink),
                                       _stream_handle(stream)), "wushkv_read_probe")
    return sink
