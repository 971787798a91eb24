"""Test-side reader of the packed page layout, written from the description
in include/wushkv.h (not from the kernels), so a layout slip on the GPU side
shows up as a parity failure rather than cancelling out.

One (page, head) block: K code words, V code words, K params, V params.
A word holds B = 32 / bits codes.
Both regions are sequences of 16-byte chunks; chunk q holds word q*4 .. q*4+3
of every lane in lane order, so a lane's k-th word is word
(k // 4) * 4 * lanes + 4 L + k % 4 of the region.
K: lane L = 16 j + n (j < d / 32; d / 2 lanes) owns 4 bits words; its word
  k = bits*t + w holds code e = h (B/2) + i (h = 0, 1; i < B/2) at
  bit 2 bits i + bits h : token 4 n + t, channel 32 j + B w + e
V: element e is slot i = e % 8 of operand o = e // 8 and sits at bit
  16 * (i % 2) + F(o, i // 2) with F = (6, 10, 8, 12 | 2, 0, 4, 14) for
  2-bit operands 0 | 1 and (4, 0, 8, 12) for 4-bit.  Lane L = 16 j + m (64
  lanes) owns 4 nw words, nw = d * bits / 128; its word k = kc*2nw + u holds
  token 32 kc + 8 j + i, channel 16 nt + m, nt = u (B/8) + o
"""
from __future__ import annotations

import functools

import numpy as np

PAGE = 64


def storage_bits(bits: int) -> int:
    """3-bit codes are stored in the 4-bit format, one per 4-bit field with
    its top bit zero (the header's description of bits = 3)."""
    return 4 if bits == 3 else bits


def page_bytes(d: int, bits: int) -> int:
    return PAGE * (2 * d * storage_bits(bits) // 8 + 8)


def _v_field(bits: int, o: int, r: int) -> int:
    """Bit of the low-half code of register r of operand o in a V word."""
    if bits == 2:
        return (6, 10, 8, 12)[r] if o == 0 else (2, 0, 4, 14)[r]
    return (4, 0, 8, 12)[r]


@functools.lru_cache(maxsize=None)
def _maps(d: int, bits: int):
    """For every (word, element): (token, channel) for K and for V, and the
    bit of each element (K and V order their elements differently)."""
    B = 32 // bits
    nw = d * bits // 128
    ops = B // 8
    n_words = 64 * 4 * nw
    kt = np.empty((n_words, B), np.int64)
    kc_ = np.empty((n_words, B), np.int64)
    vt = np.empty((n_words, B), np.int64)
    vc_ = np.empty((n_words, B), np.int64)
    kbit = np.array([2 * bits * (e % (B // 2)) + bits * (e // (B // 2)) for e in range(B)], np.int64)
    vbit = np.array([16 * (e % 2) + _v_field(bits, e // 8, (e % 8) // 2) for e in range(B)], np.int64)
    for L in range(d // 2):
        j, n = divmod(L, 16)
        for t in range(4):
            for w in range(bits):
                k = bits * t + w  # the lane's k-th word: word k % 4 of chunk k // 4
                widx = (k // 4) * 4 * (d // 2) + 4 * L + k % 4
                for e in range(B):
                    kt[widx, e] = 4 * n + t
                    kc_[widx, e] = 32 * j + B * w + e
    for L in range(64):
        j, m = divmod(L, 16)
        for kc in range(2):
            for u in range(2 * nw):
                k = kc * 2 * nw + u
                widx = (k // 4) * 256 + 4 * L + k % 4
                for e in range(B):
                    o, i = divmod(e, 8)
                    nt = u * ops + o
                    vt[widx, e] = 32 * kc + 8 * j + i
                    vc_[widx, e] = 16 * nt + m
    return kt, kc_, vt, vc_, kbit, vbit


def decode_block(block: np.ndarray, d: int, bits: int):
    """block: uint8 [page_bytes] -> (kcodes [64][d], vcodes [64][d],
    kparams [64][2], vparams [64][2]) with params as fp16 bit patterns
    (scale, zero)."""
    block = np.ascontiguousarray(block, dtype=np.uint8)
    code_bits, bits = bits, storage_bits(bits)
    region = 8 * d * bits
    kt, kch, vt, vch, kbit, vbit = _maps(d, bits)
    mask = (1 << bits) - 1
    kw = block[:region].view("<u4").astype(np.int64)
    vw = block[region:2 * region].view("<u4").astype(np.int64)
    kcodes = np.full((PAGE, d), -1, np.int64)
    vcodes = np.full((PAGE, d), -1, np.int64)
    kcodes[kt, kch] = (kw[:, None] >> kbit[None, :]) & mask
    vcodes[vt, vch] = (vw[:, None] >> vbit[None, :]) & mask
    assert (kcodes >= 0).all() and (vcodes >= 0).all(), "layout map is not a bijection"
    assert kcodes.max() < (1 << code_bits) and vcodes.max() < (1 << code_bits), "code out of range"
    prm = block[2 * region:2 * region + 8 * PAGE].view("<u2").reshape(2, PAGE, 2)
    return kcodes.astype(np.uint8), vcodes.astype(np.uint8), prm[0].copy(), prm[1].copy()


def encode_block(kcodes, vcodes, kparams, vparams, d: int, bits: int) -> np.ndarray:
    """Inverse of decode_block (used to check the maps form a bijection)."""
    bits = storage_bits(bits)
    region = 8 * d * bits
    kt, kch, vt, vch, kbit, vbit = _maps(d, bits)
    kw = (np.asarray(kcodes, np.int64)[kt, kch] << kbit[None, :]).sum(axis=1)
    vw = (np.asarray(vcodes, np.int64)[vt, vch] << vbit[None, :]).sum(axis=1)
    out = np.zeros(page_bytes(d, bits), np.uint8)
    out[:region] = kw.astype("<u4").view(np.uint8)
    out[region:2 * region] = vw.astype("<u4").view(np.uint8)
    prm = np.stack([np.asarray(kparams, np.uint16), np.asarray(vparams, np.uint16)])
    out[2 * region:] = prm.astype("<u2").reshape(-1).view(np.uint8)
    return out


def gather_sequence(pages: np.ndarray, page_table: np.ndarray, b: int, h: int, n_kv: int,
                    d: int, bits: int, s_sink: int, q_end: int):
    """Codes and params of positions [s_sink, q_end) of (sequence b, head h),
    read from a host copy of the page pool."""
    pb = page_bytes(d, bits)
    pool = pages.reshape(-1, n_kv, pb)
    n = max(0, q_end - s_sink)
    kc = np.zeros((n, d), np.uint8)
    vc = np.zeros((n, d), np.uint8)
    kp = np.zeros((n, 2), np.uint16)
    vp = np.zeros((n, 2), np.uint16)
    for lp in range((n + PAGE - 1) // PAGE):
        k1, v1, kp1, vp1 = decode_block(pool[page_table[b, lp], h], d, bits)
        lo, hi = lp * PAGE, min(n, (lp + 1) * PAGE)
        kc[lo:hi], vc[lo:hi] = k1[:hi - lo], v1[:hi - lo]
        kp[lo:hi], vp[lo:hi] = kp1[:hi - lo], vp1[:hi - lo]
    return kc, vc, kp, vp
