"""WUSH-KV CPU oracle -- test infrastructure only.

Python view of the plain C reference in ``wushkv_oracle.c``.  Only the tests,
``__graft_entry__.smoke()`` and the benchmark's ``cpu_baseline`` leg may
import this package; the GPU library and its Python binding never do, and
this package imports nothing from them.

The oracle works on a *logical* cache: per (sequence, kv-head) it keeps the
bf16 value of every position plus the codes and fp16 (scale, zero) of the
quantised positions.  It knows nothing of pages, rings or kernel layouts.

Paper references: Eq. (2) attention, Eq. (3) transform insertion, Eq. (7)
and Eq. (5) quantisers, Sec. 4.4 windows, Alg. 2 cache management, Eq. (1)
the WUSH transform.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "wushkv_oracle.c")
_LIB_PATH = os.path.join(_HERE, "_build", "liboracle.so")

_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (fp-contract off: the quantiser's fp32
    sequence must not be fused)."""
    if not force and os.path.exists(_LIB_PATH):
        return _LIB_PATH
    os.makedirs(os.path.dirname(_LIB_PATH), exist_ok=True)
    tmp = _LIB_PATH + ".tmp%d" % os.getpid()
    # -fopenmp only spreads independent (sequence, head) pairs over threads
    # (orc_*_heads_parallel); every pair's arithmetic is the serial code's
    cmd = ["gcc", "-std=c11", "-O2", "-ffp-contract=off", "-fno-fast-math", "-fopenmp",
           "-fPIC", "-shared", "-o", tmp, _SRC, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build()
        _lib = ctypes.CDLL(_LIB_PATH)
        _declare(_lib)
    return _lib


_P = ctypes.c_void_p
_I32 = ctypes.c_int32
_I64 = ctypes.c_int64
_F32 = ctypes.c_float


def _declare(L):
    L.orc_bf16_to_f32.argtypes = [ctypes.c_uint16]
    L.orc_bf16_to_f32.restype = _F32
    L.orc_f32_to_bf16.argtypes = [_F32]
    L.orc_f32_to_bf16.restype = ctypes.c_uint16
    L.orc_f32_to_f16.argtypes = [_F32]
    L.orc_f32_to_f16.restype = ctypes.c_uint16
    L.orc_f16_to_f32.argtypes = [ctypes.c_uint16]
    L.orc_f16_to_f32.restype = _F32
    for name in ("orc_f32_to_bf16_array", "orc_f32_to_f16_array",
                 "orc_f16_to_f32_array", "orc_f64_to_bf16_array"):
        getattr(L, name).argtypes = [_P, _P, _I64]
        getattr(L, name).restype = None
    L.orc_kappa_position.argtypes = [_F32, ctypes.c_int, _P, _P]
    L.orc_kappa_position.restype = None
    L.orc_quantile_abs.argtypes = [_P, ctypes.c_int, _I32, _F32]
    L.orc_quantile_abs.restype = _F32
    L.orc_quantize_groups.argtypes = [_P, _I64, ctypes.c_int, ctypes.c_int, _F32, _P, _P]
    L.orc_quantize_groups.restype = None
    L.orc_dequant.argtypes = [ctypes.c_uint8, ctypes.c_uint16, ctypes.c_uint16]
    L.orc_dequant.restype = _F32
    L.orc_next_quant_end.argtypes = [_I32] * 5
    L.orc_next_quant_end.restype = _I32
    L.orc_quest_quantize_groups.argtypes = [_P, _I64, ctypes.c_int, ctypes.c_int, _F32, _P, _P]
    L.orc_quest_quantize_groups.restype = None
    L.orc_append_head.argtypes = [ctypes.c_int] * 6 + [_F32, _F32, _F32, _I32, _I32, _I32,
                                                       _P, _I64, _P, _I64, _P,
                                                       _P, _P, _P, _P, _P, _P]
    L.orc_append_head.restype = _I32
    L.orc_attend.argtypes = [ctypes.c_int, _I64, _P, _P, _P, ctypes.c_double, _P]
    L.orc_attend.restype = None
    L.orc_decode_head.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, _I32, _I32,
                                  _P, _P, _P, _P, _P, _P, _P, _P, _F32, _P]
    L.orc_decode_head.restype = None
    L.orc_decode_heads_parallel.argtypes = [ctypes.c_int] * 5 + [_P] * 10 + [_F32, _P]
    L.orc_decode_heads_parallel.restype = ctypes.c_int
    L.orc_append_heads_parallel.argtypes = [ctypes.c_int] * 8 + [_F32] * 3 + [_P] * 13
    L.orc_append_heads_parallel.restype = ctypes.c_int


def _ptr(a: np.ndarray):
    assert a.flags["C_CONTIGUOUS"], "oracle arrays must be C-contiguous"
    return a.ctypes.data_as(ctypes.c_void_p)


# --------------------------------------------------------------------------
# Number formats
# --------------------------------------------------------------------------

def _conv(x, in_dtype, out_dtype, fn_name):
    a = np.asarray(x, dtype=in_dtype)
    flat = np.ascontiguousarray(a.reshape(-1))
    y = np.empty(flat.shape, dtype=out_dtype)
    getattr(lib(), fn_name)(_ptr(flat), _ptr(y), flat.size)
    return y.reshape(a.shape)


def f32_to_bf16(x) -> np.ndarray:
    """fp32 -> bf16 bit patterns (uint16), round to nearest even."""
    return _conv(x, np.float32, np.uint16, "orc_f32_to_bf16_array")


def f64_to_bf16(x) -> np.ndarray:
    """fp64 -> bf16 bit patterns in a single rounding."""
    return _conv(x, np.float64, np.uint16, "orc_f64_to_bf16_array")


def bf16_to_f32(h) -> np.ndarray:
    a = np.asarray(h, dtype=np.uint16)
    return (a.astype(np.uint32) << 16).view(np.float32)


def f32_to_f16(x) -> np.ndarray:
    """fp32 -> fp16 bit patterns (uint16), round to nearest even."""
    return _conv(x, np.float32, np.uint16, "orc_f32_to_f16_array")


def f16_to_f32(h) -> np.ndarray:
    return _conv(h, np.uint16, np.float32, "orc_f16_to_f32_array")


# --------------------------------------------------------------------------
# Quantiser, Eq. (7)
# --------------------------------------------------------------------------

def kappa_position(kappa: float, d: int):
    lo = ctypes.c_int32()
    t = ctypes.c_float()
    lib().orc_kappa_position(kappa, d, ctypes.byref(lo), ctypes.byref(t))
    return lo.value, t.value


def quantile_abs(x, kappa: float) -> float:
    x = np.ascontiguousarray(x, dtype=np.float32)
    lo, t = kappa_position(kappa, x.size)
    return lib().orc_quantile_abs(_ptr(x), x.size, lo, t)


def quantize_groups(x, bits: int, kappa: float):
    """x [..., d] fp32 -> (codes uint8 [..., d], scale16 uint16 [...], zero16 uint16 [...])."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    d = x.shape[-1]
    n = x.size // d
    codes = np.empty(x.shape, dtype=np.uint8)
    params = np.empty(x.shape[:-1] + (2,), dtype=np.uint16)
    lib().orc_quantize_groups(_ptr(x), n, d, bits, kappa, _ptr(codes), _ptr(params))
    return codes, params[..., 0].copy(), params[..., 1].copy()


# --------------------------------------------------------------------------
# QuEST quantiser, Eq. (5)
# --------------------------------------------------------------------------

def quest_grid_mse(alpha: float, bits: int) -> float:
    """Mean squared error of rounding a standard Gaussian to the nearest of
    the 2^bits levels spaced evenly from -alpha to +alpha (Sec. 4.3, and the
    fixed-scale grid of the clipping lemma in App. B).  Sum over the levels
    of the integral of (x - level)^2 over its nearest-level cell, with the
    Gaussian moments int phi = Phi, int x phi = -phi, int x^2 phi = Phi - x phi."""
    from scipy.special import ndtr
    n = 1 << bits
    lv = -alpha + 2.0 * alpha / (n - 1) * np.arange(n, dtype=np.float64)
    edges = np.concatenate([[-np.inf], 0.5 * (lv[1:] + lv[:-1]), [np.inf]])
    a, b = edges[:-1], edges[1:]
    phi = lambda t: np.where(np.isfinite(t), np.exp(-0.5 * np.where(np.isfinite(t), t, 0.0) ** 2)
                             / np.sqrt(2.0 * np.pi), 0.0)
    tphi = lambda t: np.where(np.isfinite(t), np.where(np.isfinite(t), t, 0.0) * phi(t), 0.0)
    m0 = ndtr(b) - ndtr(a)
    m1 = phi(a) - phi(b)
    m2 = m0 - (tphi(b) - tphi(a))
    return float(np.sum(m2 - 2.0 * lv * m1 + lv * lv * m0))


def quest_alpha(bits: int) -> float:
    """alpha_b of Eq. (5): the endpoint that minimises quest_grid_mse (Sec. 4.3),
    found by bounded scalar minimisation of the error itself."""
    from scipy.optimize import minimize_scalar
    r = minimize_scalar(lambda a: quest_grid_mse(a, bits), bounds=(1e-3, 16.0), method="bounded",
                        options={"xatol": 1e-12, "maxiter": 500})
    return float(r.x)


def quest_quantize_groups(x, bits: int, alpha: float):
    """x [..., d] fp32 -> (codes uint8 [..., d] in [0, 2^bits - 1],
    scale16, zero16 uint16 [...]) of Eq. (5); reconstruction is
    dequant(codes, scale16, zero16)."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    d = x.shape[-1]
    n = x.size // d
    codes = np.empty(x.shape, dtype=np.uint8)
    params = np.empty(x.shape[:-1] + (2,), dtype=np.uint16)
    lib().orc_quest_quantize_groups(_ptr(x), n, d, bits, alpha, _ptr(codes), _ptr(params))
    return codes, params[..., 0].copy(), params[..., 1].copy()


def dequant(codes, s16, z16) -> np.ndarray:
    """fp32 reconstruction scale * code + zero (one rounding)."""
    codes = np.asarray(codes, dtype=np.uint8)
    s = f16_to_f32(np.asarray(s16, dtype=np.uint16))[..., None]
    z = f16_to_f32(np.asarray(z16, dtype=np.uint16))[..., None]
    # s * code is exact in fp32 (11-bit significand times a <= 4-bit integer),
    # so the fp64 sum rounded once to fp32 equals fmaf(s, code, z).
    return (s.astype(np.float64) * codes + z.astype(np.float64)).astype(np.float32)


# --------------------------------------------------------------------------
# Windows and bookkeeping, Sec. 4.4 / Alg. 2
# --------------------------------------------------------------------------

def next_quant_end(s_new: int, s_quant: int, s_sink: int, s_keep: int, s_flush: int) -> int:
    return lib().orc_next_quant_end(s_new, s_quant, s_sink, s_keep, s_flush)


class OracleCache:
    """Logical WUSH-KV cache for ``batch`` sequences and ``n_kv`` heads.

    Holds, per (sequence, head), the bf16 pattern of every cached position and
    the codes / fp16 params of the quantised ones.  ``append`` follows Alg. 2
    steps 3-4 and 7-11; ``decode`` follows Eq. (2) with the Eq. (3) query
    compensation.
    """

    def __init__(self, batch, n_kv, d, bits, s_sink, s_keep, s_flush,
                 kappa_k, kappa_v, capacity, codec="pclip", quest_alpha=0.0):
        self.batch, self.n_kv, self.d, self.bits = batch, n_kv, d, bits
        self.s_sink, self.s_keep, self.s_flush = s_sink, s_keep, s_flush
        self.kappa_k, self.kappa_v = float(kappa_k), float(kappa_v)
        assert codec in ("pclip", "quest")
        self.codec, self.quest_alpha = codec, float(quest_alpha)
        self.cap = capacity
        shp = (batch, n_kv, capacity, d)
        self.kbits = np.zeros(shp, np.uint16)
        self.vbits = np.zeros(shp, np.uint16)
        self.kc = np.zeros(shp, np.uint8)
        self.vc = np.zeros(shp, np.uint8)
        self.kp = np.zeros((batch, n_kv, capacity, 2), np.uint16)
        self.vp = np.zeros((batch, n_kv, capacity, 2), np.uint16)
        self.seq_len = np.zeros(batch, np.int32)
        self.quant_end = np.zeros(batch, np.int32)

    def append(self, k_new, v_new, n_new, tk):
        """k_new, v_new: bf16 patterns [batch][max_new][n_kv][d];
        n_new: [batch] ints; tk: bf16 patterns [n_kv][d][d] (k~ = T_K k)."""
        k_new = np.ascontiguousarray(k_new, dtype=np.uint16)
        v_new = np.ascontiguousarray(v_new, dtype=np.uint16)
        tk = np.ascontiguousarray(tk, dtype=np.uint16)
        L = lib()
        d, nkv = self.d, self.n_kv
        row_stride = nkv * d
        for b in range(self.batch):
            n = int(n_new[b])
            s_old, q_old = int(self.seq_len[b]), int(self.quant_end[b])
            assert s_old + n <= self.cap, "oracle cache capacity exceeded"
            q_new = q_old
            for h in range(nkv):
                # pointer to (b, token 0, head h); token rows are row_stride apart
                kptr = ctypes.c_void_p(k_new.ctypes.data + (b * k_new.shape[1] * nkv + h) * d * 2)
                vptr = ctypes.c_void_p(v_new.ctypes.data + (b * v_new.shape[1] * nkv + h) * d * 2)
                q_new = L.orc_append_head(
                    d, self.bits, self.s_sink, self.s_keep, self.s_flush,
                    1 if self.codec == "quest" else 0, self.kappa_k, self.kappa_v,
                    self.quest_alpha, s_old, q_old, n,
                    kptr, row_stride, vptr, row_stride,
                    _ptr(tk[h]),
                    _ptr(self.kbits[b, h]), _ptr(self.vbits[b, h]),
                    _ptr(self.kc[b, h]), _ptr(self.kp[b, h]),
                    _ptr(self.vc[b, h]), _ptr(self.vp[b, h]))
            self.seq_len[b] = s_old + n
            self.quant_end[b] = q_new

    def decode(self, q, tinv, sm_scale, heads=None):
        """q: bf16 patterns [batch][n_q][d]; tinv: fp32 [n_kv][d][d].
        Returns fp64 [batch][n_q][d].  ``heads`` optionally restricts the work
        to a list of (b, h) pairs (other rows are left NaN)."""
        q = np.ascontiguousarray(q, dtype=np.uint16)
        tinv = np.ascontiguousarray(tinv, dtype=np.float32)
        nq = q.shape[1]
        G = nq // self.n_kv
        out = np.full((self.batch, nq, self.d), np.nan, np.float64)
        pairs = heads if heads is not None else [(b, h) for b in range(self.batch)
                                                 for h in range(self.n_kv)]
        for b, h in pairs:
            o = np.empty((G, self.d), np.float64)
            qg = np.ascontiguousarray(q[b, h * G:(h + 1) * G])
            decode_head(self.d, G, self.s_sink, int(self.seq_len[b]), int(self.quant_end[b]),
                        self.kbits[b, h], self.vbits[b, h], self.kc[b, h], self.kp[b, h],
                        self.vc[b, h], self.vp[b, h], qg, tinv[h], sm_scale, o)
            out[b, h * G:(h + 1) * G] = o
        return out


def decode_step(cache: "OracleCache", k_new, v_new, n_new, tk, q, tinv, sm_scale):
    """One decode step of Alg. 2 (S' = 1) in the algorithm's own order: the
    new tokens are appended in full precision (steps 3-4), attention runs
    over the cache (step 5), and only then are the positions that left the
    recent window quantised (steps 7-11).  So step 5 sees those positions at
    bf16.  k_new, v_new: bf16 patterns [batch][n_kv][d]; n_new: [batch] of 0
    or 1.  Returns fp64 [batch][n_q][d]; the cache ends as after append."""
    k_new = np.ascontiguousarray(k_new, dtype=np.uint16)[:, None]
    v_new = np.ascontiguousarray(v_new, dtype=np.uint16)[:, None]
    q_before = cache.quant_end.copy()
    # append() quantises as well, but it keeps every position's bf16 pattern,
    # and decode() reads the patterns of positions at or after quant_end: the
    # attention of step 5 is decode() with the boundary from before the flush
    cache.append(k_new, v_new, n_new, tk)
    q_after = cache.quant_end.copy()
    cache.quant_end[:] = q_before
    try:
        out = cache.decode(q, tinv, sm_scale)
    finally:
        cache.quant_end[:] = q_after
    return out


def chunk_attention(cache: "OracleCache", q, n_tok, tinv, sm_scale):
    """Attention of a chunk of new tokens (Alg. 2 step 5 with S' > 1; the
    causal mask of Eq. (2)): q bf16 patterns [batch][S'][n_q][d]; sequence b's
    chunk is its last n_tok[b] positions, token t at position
    p = seq_len[b] - n_tok[b] + t, which attends to positions [0, p].  Rows
    t >= n_tok[b] are left NaN.  Returns fp64 [batch][S'][n_q][d]."""
    q = np.ascontiguousarray(q, dtype=np.uint16)
    tinv = np.ascontiguousarray(tinv, dtype=np.float32)
    B, T, nq, d = q.shape
    G = nq // cache.n_kv
    out = np.full((B, T, nq, d), np.nan, np.float64)
    for b in range(B):
        S, Q = int(cache.seq_len[b]), int(cache.quant_end[b])
        n = int(n_tok[b])
        for t in range(n):
            visible = S - n + t + 1  # positions [0, visible)
            for h in range(cache.n_kv):
                o = np.empty((G, d), np.float64)
                qg = np.ascontiguousarray(q[b, t, h * G:(h + 1) * G])
                decode_head(d, G, cache.s_sink, visible, min(Q, visible), cache.kbits[b, h],
                            cache.vbits[b, h], cache.kc[b, h], cache.kp[b, h], cache.vc[b, h],
                            cache.vp[b, h], qg, tinv[h], sm_scale, o)
                out[b, t, h * G:(h + 1) * G] = o
    return out


def decode_head(d, G, s_sink, S, q_end, kbits, vbits, kc, kp, vc, vp, q, tinv, sm_scale, out):
    """Thin wrapper over orc_decode_head; arrays are per (sequence, head):
    kbits/vbits [cap][d] uint16, kc/vc [cap][d] uint8, kp/vp [cap][2] uint16,
    q [G][d] uint16 (bf16), tinv [d][d] fp32, out [G][d] fp64 (written)."""
    args = [np.ascontiguousarray(a) for a in (kbits, vbits, kc, kp, vc, vp, q, tinv)]
    assert out.flags["C_CONTIGUOUS"] and out.dtype == np.float64
    lib().orc_decode_head(d, G, s_sink, S, q_end, *[_ptr(a) for a in args],
                          float(sm_scale), _ptr(out))
    return out


def _ptr_array(arrays):
    return (ctypes.c_void_p * len(arrays))(*[a.ctypes.data for a in arrays])


class HeadSet:
    """Logical caches of independent (sequence, kv head) pairs for the
    benchmark's CPU baseline: each pair is a one-sequence, one-head cache of
    capacity ``caps[i]``, filled and decoded with orc_append_head and
    orc_decode_head, the pairs spread over host threads (OpenMP).  Only the
    threading differs from OracleCache; every pair's arithmetic is the same."""

    def __init__(self, caps, d, bits, s_sink, s_keep, s_flush, kappa_k, kappa_v):
        self.d, self.bits = d, bits
        self.s_sink, self.s_keep, self.s_flush = s_sink, s_keep, s_flush
        self.kappa_k, self.kappa_v = float(kappa_k), float(kappa_v)
        self.caps = [int(c) for c in caps]
        n = len(self.caps)
        self.kbits = [np.zeros((c, d), np.uint16) for c in self.caps]
        self.vbits = [np.zeros((c, d), np.uint16) for c in self.caps]
        self.kc = [np.zeros((c, d), np.uint8) for c in self.caps]
        self.vc = [np.zeros((c, d), np.uint8) for c in self.caps]
        self.kp = [np.zeros((c, 2), np.uint16) for c in self.caps]
        self.vp = [np.zeros((c, 2), np.uint16) for c in self.caps]
        self.seq_len = np.zeros(n, np.int32)
        self.quant_end = np.zeros(n, np.int32)

    def append(self, k_new, v_new, tk, threads=0):
        """k_new[i], v_new[i]: bf16 patterns [n_i][d] of pair i; tk[i]: bf16
        [d][d].  Returns the threads used."""
        n = len(self.caps)
        k_new = [np.ascontiguousarray(k, np.uint16) for k in k_new]
        v_new = [np.ascontiguousarray(v, np.uint16) for v in v_new]
        tk = [np.ascontiguousarray(t, np.uint16) for t in tk]
        n_new = np.array([k.shape[0] for k in k_new], np.int32)
        assert np.all(self.seq_len + n_new <= np.array(self.caps)), "capacity exceeded"
        q_new = np.zeros(n, np.int32)
        used = lib().orc_append_heads_parallel(
            n, threads, self.d, self.bits, self.s_sink, self.s_keep, self.s_flush, 0,
            self.kappa_k, self.kappa_v, 0.0, _ptr(self.seq_len.copy()), _ptr(self.quant_end.copy()),
            _ptr(n_new), _ptr_array(k_new), _ptr_array(v_new), _ptr_array(tk),
            _ptr_array(self.kbits), _ptr_array(self.vbits), _ptr_array(self.kc),
            _ptr_array(self.kp), _ptr_array(self.vc), _ptr_array(self.vp), _ptr(q_new))
        self.seq_len += n_new
        self.quant_end[:] = q_new
        return used

    def decode(self, q, tinv, sm_scale, threads=0, pairs=None):
        """q[i]: bf16 patterns [G][d] of pair i; tinv[i]: fp32 [d][d].
        Returns (fp64 outputs [n][G][d], threads used).  ``pairs`` restricts
        the call to those indices."""
        idx = list(range(len(self.caps))) if pairs is None else list(pairs)
        q = [np.ascontiguousarray(q[i], np.uint16) for i in idx]
        tinv = [np.ascontiguousarray(tinv[i], np.float32) for i in idx]
        G = q[0].shape[0]
        out = [np.empty((G, self.d), np.float64) for _ in idx]
        S = np.ascontiguousarray(self.seq_len[idx])
        Q = np.ascontiguousarray(self.quant_end[idx])
        pick = lambda arrs: _ptr_array([arrs[i] for i in idx])
        used = lib().orc_decode_heads_parallel(
            len(idx), threads, self.d, G, self.s_sink, _ptr(S), _ptr(Q), pick(self.kbits),
            pick(self.vbits), pick(self.kc), pick(self.kp), pick(self.vc), pick(self.vp),
            _ptr_array(q), _ptr_array(tinv), float(sm_scale), _ptr_array(out))
        return np.stack(out), used


def attend(q, K, V, scale: float) -> np.ndarray:
    """fp64 softmax attention of one query q [d] over K, V [S][d]."""
    q = np.ascontiguousarray(q, dtype=np.float64)
    K = np.ascontiguousarray(K, dtype=np.float64)
    V = np.ascontiguousarray(V, dtype=np.float64)
    d = q.shape[0]
    out = np.empty(d, np.float64)
    lib().orc_attend(d, K.shape[0], _ptr(q), _ptr(K), _ptr(V), float(scale), _ptr(out))
    return out


# --------------------------------------------------------------------------
# Headwise normalisation and rotary embedding of new keys (Eq. (2), Alg. 2
# step 1; the RMS form of Norm and the pairwise rotations R_s of RoPE are
# those written in the appendix on RoPE-commuting transforms)
# --------------------------------------------------------------------------

def rope_frequencies(theta: float, d: int) -> np.ndarray:
    """omega_j = theta^(-2j/d) for the d/2 rotary pairs, fp64."""
    return float(theta) ** (-2.0 * np.arange(d // 2, dtype=np.float64) / d)


def norm_rope(k_bits, positions, theta: float, gain=None, eps: float = 0.0) -> np.ndarray:
    """bf16 patterns of RoPE(Norm(k)) for keys k (bf16 patterns [..., n, d])
    at integer positions [n], evaluated in fp64 and rounded once to bf16.

    Norm(x) = diag(gain) x / sqrt(mean_i x_i^2 + eps): the RMS normalisation
    d^(1/2) ||x||^-1 diag(gain) x, with eps inside the root (eps = 0 is the
    form written in the paper).  RoPE rotates coordinate pair (j, j + d/2)
    by the angle s omega_j of position s: the 2x2 rotation
    [[cos, -sin], [sin, cos]] applied to (x_j, x_{j+d/2})."""
    x = bf16_to_f32(np.asarray(k_bits, np.uint16)).astype(np.float64)
    d = x.shape[-1]
    half = d // 2
    ms = np.mean(x * x, axis=-1, keepdims=True)
    g = np.ones(d) if gain is None else np.asarray(gain, np.float64)
    y = x / np.sqrt(ms + float(eps)) * g
    ang = np.asarray(positions, np.float64)[:, None] * rope_frequencies(theta, d)[None, :]
    shape = (1,) * (x.ndim - 2) + ang.shape
    c = np.cos(ang).reshape(shape)
    s = np.sin(ang).reshape(shape)
    y1, y2 = y[..., :half], y[..., half:]
    out = np.concatenate([y1 * c - y2 * s, y2 * c + y1 * s], axis=-1)
    return f64_to_bf16(out)


# --------------------------------------------------------------------------
# The WUSH transform, Eq. (1) (Sec. 3; used per head by Eq. (4) and Alg. 1)
# --------------------------------------------------------------------------

def sylvester_hadamard(d: int) -> np.ndarray:
    """The normalised Hadamard matrix of order d = 2^m in Sylvester's order:
    entry (i, j) is (-1)^popcount(i & j) / sqrt(d)."""
    i = np.arange(d)
    bits = np.bitwise_and(i[:, None], i[None, :])
    sign = np.ones((d, d))
    for b in range(int(np.log2(d))):
        sign *= np.where((bits >> b) & 1, -1.0, 1.0)
    return sign / np.sqrt(d)


def wush_transform(M, H, gamma: float):
    """T = Wush(M, H, gamma) of Eq. (1) in fp64, with T^{-1}:
      L L^T = H + gamma tr(H)/d I                 (Cholesky, L lower)
      U Lam U^T = L^T (M + gamma tr(M)/d I) L     (symmetric eigendecomposition)
      c = (1 + gamma)^(1/2) tr(M)^(1/2) tr(Lam^(1/2))^(-1/2)
      T = c Had Lam^(-1/4) U^T L^T
    The eigendecomposition is unique only up to the order of the eigenpairs
    and the sign of each eigenvector, and Had mixes them, so T depends on
    both.  The paper fixes neither; this reading takes the eigenvalues in
    ascending order and the sign of u_k that makes the largest-magnitude
    entry of L u_k positive (the first such entry on a tie), with the
    Hadamard matrix in Sylvester's order.  Returns (T, T^{-1}, Lam)."""
    M = np.asarray(M, np.float64)
    H = np.asarray(H, np.float64)
    d = M.shape[0]
    I = np.eye(d)
    L = np.linalg.cholesky(H + gamma * np.trace(H) / d * I)
    S = L.T @ (M + gamma * np.trace(M) / d * I) @ L
    lam, U = np.linalg.eigh(0.5 * (S + S.T))   # ascending
    W = L @ U
    for k in range(d):
        i = int(np.argmax(np.abs(W[:, k])))
        if W[i, k] < 0:
            U[:, k] = -U[:, k]
            W[:, k] = -W[:, k]
    c = np.sqrt(1.0 + gamma) * np.sqrt(np.trace(M)) / np.sqrt(np.sum(np.sqrt(lam)))
    Had = sylvester_hadamard(d)
    T = c * Had @ np.diag(lam ** -0.25) @ U.T @ L.T
    return T, np.linalg.inv(T), lam
