"""Drive the GPU library and the oracle side by side on the same inputs.

A ``Pair`` holds one GPU cache and two oracle caches:
  ref     fed the raw inputs; applies T_K itself in fp64;
  mirror  fed the GPU's own transformed keys k~ (with T = I, which the
          oracle applies exactly), so its codes, params, windows and
          counters must equal the GPU's bit for bit.
Comparisons read the GPU pages with the test-side decoder (pagelayout.py).
"""
from __future__ import annotations

import sys

import numpy as np
import torch

import oracle
import pagelayout
import paper_2609_38121_amd as wk
from workloads import synth

TOL = 2e-3  # max relative error of decode outputs, row-normalised


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def to_dev_bf16(bits: np.ndarray, dev) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(dev).view(torch.bfloat16)


def to_np_bits(t: torch.Tensor) -> np.ndarray:
    return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def rel_err(gpu: np.ndarray, ref: np.ndarray) -> float:
    """max over rows of ||gpu - ref||_inf / max(||ref||_inf, 1e-6)."""
    g = gpu.reshape(-1, gpu.shape[-1]).astype(np.float64)
    r = ref.reshape(-1, ref.shape[-1]).astype(np.float64)
    num = np.max(np.abs(g - r), axis=1)
    den = np.maximum(np.max(np.abs(r), axis=1), 1e-6)
    return float(np.max(num / den))


def eye_bits(n_kv: int, d: int) -> np.ndarray:
    return oracle.f32_to_bf16(np.broadcast_to(np.eye(d, dtype=np.float32), (n_kv, d, d)).copy())


def tie_patched(ref: oracle.OracleCache, mirror: oracle.OracleCache):
    """The end-to-end reference cache ``ref`` (T_K applied in fp64 to the raw
    keys) with one change: every position whose key codes differ from the
    GPU's (the mirror's) takes the GPU's bf16 k~ row instead of the fp64 one.
    Those are the positions where the fp32-accumulated k~ rounded to the
    other bf16 neighbour of a code decision's tie, so the returned cache
    differs from ``ref`` exactly there and nowhere else.  Returns (cache,
    number of substituted positions)."""
    B, H, d = ref.batch, ref.n_kv, ref.d
    out = oracle.OracleCache(B, H, d, ref.bits, ref.s_sink, ref.s_keep, ref.s_flush, ref.kappa_k,
                             ref.kappa_v, ref.cap, codec=ref.codec, quest_alpha=ref.quest_alpha)
    S = ref.seq_len.astype(np.int64)
    n = max(1, int(S.max()))
    k = np.zeros((B, n, H, d), np.uint16)
    v = np.zeros_like(k)
    subst = 0
    for b in range(B):
        qe = max(int(ref.quant_end[b]), ref.s_sink)
        for h in range(H):
            kb = ref.kbits[b, h, :S[b]].copy()
            if qe > ref.s_sink:
                sl = slice(ref.s_sink, qe)
                rows = ref.s_sink + np.nonzero(np.any(ref.kc[b, h, sl] != mirror.kc[b, h, sl], axis=1))[0]
                kb[rows] = mirror.kbits[b, h, rows]
                subst += len(rows)
            k[b, :S[b], h] = kb
            v[b, :S[b], h] = ref.vbits[b, h, :S[b]]
    out.append(k, v, S.astype(np.int32), eye_bits(H, d))
    assert np.array_equal(out.quant_end, ref.quant_end)
    # every key code now equals the GPU's: the reference's where they agreed,
    # the GPU's own k~ where they did not
    for b in range(B):
        qe = max(int(ref.quant_end[b]), ref.s_sink)
        assert np.array_equal(out.kc[b, :, ref.s_sink:qe], mirror.kc[b, :, ref.s_sink:qe])
    return out, subst


class Pair:
    def __init__(self, dev, batch, n_kv, G, d, bits, s_sink, s_keep, s_flush, kappa_k, kappa_v,
                 cap, win_slots=None, page_order="linear", pool_factor=1.0, symmetric=True,
                 seed=0, oracle_ref=True, codec="pclip", quest_alpha="oracle"):
        """quest_alpha (QuEST caches): "oracle" gives the descriptor the
        oracle's alpha_b, None the library's default (wushkv_quest_alpha);
        the oracle caches always take the value the descriptor holds."""
        self.dev = dev
        self.batch, self.n_kv, self.G, self.d, self.bits = batch, n_kv, G, d, bits
        self.s_sink = s_sink
        if codec != "quest":
            quest_alpha = None
        elif quest_alpha == "oracle":
            quest_alpha = oracle.quest_alpha(bits)
        self.gpu = wk.WushKVCache(batch, n_kv, d, bits, s_sink, s_keep, s_flush, kappa_k,
                                  kappa_v, max_seq_len=cap, win_slots=win_slots,
                                  page_order=page_order, pool_factor=pool_factor, seed=seed,
                                  device=dev, codec=codec, quest_alpha=quest_alpha)
        args = (batch, n_kv, d, bits, s_sink, s_keep, s_flush, kappa_k, kappa_v, cap)
        # the oracle gets the clip multiplier exactly as the descriptor holds it
        kw = dict(codec=codec, quest_alpha=self.gpu.quest_alpha)
        self.ref = oracle.OracleCache(*args, **kw) if oracle_ref else None
        self.mirror = oracle.OracleCache(*args, **kw)
        self.tk, self.tinv = synth.make_transform(n_kv, d, seed, symmetric)
        self.eye = eye_bits(n_kv, d)
        self.tk_dev = to_dev_bf16(self.tk, dev)
        self.tinv_dev = torch.from_numpy(self.tinv).to(dev)
        self.sm_scale = 1.0 / np.sqrt(d)
        self.k_tilde_log = []

    # ------------------------------------------------------------ append
    def append(self, k: np.ndarray, v: np.ndarray, n_new) -> np.ndarray:
        n_new = np.asarray(n_new, np.int32)
        kd, vd = to_dev_bf16(k, self.dev), to_dev_bf16(v, self.dev)
        nd = torch.from_numpy(n_new).to(self.dev)
        kt = torch.full_like(kd, float("nan"))
        wk.wushkv_append(self.gpu, kd, vd, nd, self.tk_dev, k_tilde_out=kt)
        torch.cuda.synchronize()
        kt_np = to_np_bits(kt)
        if self.ref is not None:
            self.ref.append(k, v, n_new, self.tk)
        self.mirror.append(kt_np, v, n_new, self.eye)
        self.k_tilde_log.append((k, kt_np, n_new))
        return kt_np

    def append_norm_rope(self, k_raw: np.ndarray, v: np.ndarray, n_new, theta: float,
                         gain=None, eps: float = 1e-6) -> np.ndarray:
        """The fused append: raw keys are normalised and rotated on the GPU
        (rotary table built by the input generator); the reference oracle
        gets RoPE(Norm(k)) from the oracle's own fp64 evaluation, the mirror
        gets the GPU's k~."""
        n_new = np.asarray(n_new, np.int32)
        cap = self.gpu.max_pages * 64 + self.s_sink
        table = torch.from_numpy(synth.rope_table(theta, self.d, cap)).to(self.dev)
        g = None if gain is None else torch.from_numpy(np.asarray(gain, np.float32)).to(self.dev)
        kd, vd = to_dev_bf16(k_raw, self.dev), to_dev_bf16(v, self.dev)
        nd = torch.from_numpy(n_new).to(self.dev)
        kt = torch.full_like(kd, float("nan"))
        wk.wushkv_append_norm_rope(self.gpu, kd, vd, nd, self.tk_dev, table, norm_gain=g,
                                   norm_eps=eps, k_tilde_out=kt)
        torch.cuda.synchronize()
        kt_np = to_np_bits(kt)
        k_rot = np.zeros_like(k_raw)
        for b in range(self.batch):
            n = int(n_new[b])
            if n == 0:
                continue
            pos = int(self.mirror.seq_len[b]) + np.arange(n)
            rows = np.transpose(k_raw[b, :n], (1, 0, 2))               # [H][n][d]
            k_rot[b, :n] = np.transpose(oracle.norm_rope(rows, pos, theta, gain, eps), (1, 0, 2))
        if self.ref is not None:
            self.ref.append(k_rot, v, n_new, self.tk)
        self.mirror.append(kt_np, v, n_new, self.eye)
        self.k_tilde_log.append((k_rot, kt_np, n_new))
        return kt_np

    def step(self, k: np.ndarray, v: np.ndarray, n_new, q: np.ndarray, tol=TOL, max_seq_len=None):
        """The fused decode step (wushkv_decode_step) against the oracle's
        decode_step in Alg. 2's order: k, v bf16 patterns [batch][n_kv][d],
        n_new [batch] of 0 / 1, q [batch][n_q][d].  The mirror gets the GPU's
        k~, read back from the window slot the step wrote.  Returns (gpu
        output, error vs mirror, error vs reference)."""
        n_new = np.asarray(n_new, np.int32)
        s_old = self.mirror.seq_len.copy()
        nd = torch.from_numpy(n_new).to(self.dev)
        out = wk.wushkv_decode_step(self.gpu, to_dev_bf16(k, self.dev), to_dev_bf16(v, self.dev), nd,
                                    self.tk_dev, to_dev_bf16(q, self.dev), self.tinv_dev,
                                    sm_scale=self.sm_scale, max_seq_len=max_seq_len)
        torch.cuda.synchronize()
        gpu = out.cpu().numpy()
        win_k = to_np_bits(self.gpu.win_k)
        ring = self.gpu.win_slots - self.s_sink
        kt = np.zeros_like(k)
        for b in range(self.batch):
            if n_new[b]:
                p = int(s_old[b])
                slot = p if p < self.s_sink else self.s_sink + (p - self.s_sink) % ring
                kt[b] = win_k[b, :, slot]
        mir = oracle.decode_step(self.mirror, kt, v, n_new, self.eye, q, self.tinv, self.sm_scale)
        e_m = rel_err(gpu, mir)
        e_r = 0.0
        if self.ref is not None:
            ref = oracle.decode_step(self.ref, k, v, n_new, self.tk, q, self.tinv, self.sm_scale)
            e_r = rel_err(gpu, ref)
        self.k_tilde_log.append((k[:, None], kt[:, None], n_new))
        assert np.all(np.isfinite(gpu))
        assert e_m <= tol, "step vs oracle on the GPU's cache: %.3e" % e_m
        assert e_r <= tol, "step vs oracle from raw inputs: %.3e" % e_r
        return gpu, e_m, e_r

    def k_tilde_vs_ref(self):
        """Check the GPU's bf16 k~ = T_K k against the exact product.  The GPU
        accumulates in fp32 and rounds once to bf16, so each element must lie
        within one bf16 ulp of the exact value plus the fp32 dot-product error
        bound d 2^-24 sum_i |T_oi k_i|.  Returns (entries, entries that differ
        from the correctly rounded bf16, entries outside the bound)."""
        total = diff = bad = 0
        T = oracle.bf16_to_f32(self.tk).astype(np.float64)                 # [H][d][d]
        for k, kt, n_new in self.k_tilde_log:
            for b in range(self.batch):
                n = int(n_new[b])
                if n == 0:
                    continue
                kf = oracle.bf16_to_f32(k[b, :n]).astype(np.float64)       # [n][H][d]
                exact = np.einsum("hoi,thi->tho", T, kf)
                absum = np.einsum("hoi,thi->tho", np.abs(T), np.abs(kf))
                rb = oracle.f64_to_bf16(exact)
                g = oracle.bf16_to_f32(kt[b, :n]).astype(np.float64)
                ulp = np.abs(oracle.bf16_to_f32(rb).astype(np.float64)) * 2.0 ** -7 + 2.0 ** -133
                bound = ulp + self.d * 2.0 ** -24 * absum
                total += exact.size
                diff += int(np.count_nonzero(rb != kt[b, :n]))
                bad += int(np.count_nonzero(np.abs(g - exact) > bound))
        return total, diff, bad

    # ------------------------------------------------------------ state
    def host_state(self):
        g = self.gpu
        return (g.pages.cpu().numpy(), g.page_table.cpu().numpy(), to_np_bits(g.win_k),
                to_np_bits(g.win_v), g.seq_len.cpu().numpy(), g.quant_end.cpu().numpy())

    def check_cache(self, heads=None):
        """GPU cache == mirror (bit-exact): counters, codes, params, windows.
        Returns the number of compared codes."""
        pages, table, win_k, win_v, seq_len, quant_end = self.host_state()
        m = self.mirror
        assert np.array_equal(seq_len, m.seq_len), (seq_len, m.seq_len)
        assert np.array_equal(quant_end, m.quant_end), (quant_end, m.quant_end)
        if self.ref is not None:
            assert np.array_equal(self.ref.quant_end, m.quant_end)
        W = self.gpu.win_slots
        ring = W - self.s_sink
        n_codes = 0
        pairs = heads or [(b, h) for b in range(self.batch) for h in range(self.n_kv)]
        for b, h in pairs:
            S, Q = int(seq_len[b]), int(quant_end[b])
            qe = max(Q, self.s_sink)
            if qe > self.s_sink:
                kc, vc, kp, vp = pagelayout.gather_sequence(
                    pages, table, b, h, self.n_kv, self.d, self.bits, self.s_sink, qe)
                sl = slice(self.s_sink, qe)
                assert np.array_equal(kc, m.kc[b, h, sl]), "K codes differ (b=%d h=%d)" % (b, h)
                assert np.array_equal(vc, m.vc[b, h, sl]), "V codes differ (b=%d h=%d)" % (b, h)
                assert np.array_equal(kp, m.kp[b, h, sl]), "K params differ (b=%d h=%d)" % (b, h)
                assert np.array_equal(vp, m.vp[b, h, sl]), "V params differ (b=%d h=%d)" % (b, h)
                n_codes += 2 * kc.size
            for p in list(range(min(S, self.s_sink))) + list(range(qe, S)):
                slot = p if p < self.s_sink else self.s_sink + (p - self.s_sink) % ring
                assert np.array_equal(win_k[b, h, slot], m.kbits[b, h, p]), ("win_k", b, h, p)
                assert np.array_equal(win_v[b, h, :, slot], m.vbits[b, h, p]), ("win_v", b, h, p)
        return n_codes

    # ------------------------------------------------------------ decode
    def decode(self, q: np.ndarray, max_seq_len=None):
        qd = to_dev_bf16(q, self.dev)
        out = wk.wushkv_decode_attention(self.gpu, qd, self.tinv_dev, sm_scale=self.sm_scale,
                                         max_seq_len=max_seq_len)
        torch.cuda.synchronize()
        return out.cpu().numpy()

    def decode_check(self, q: np.ndarray, tol=TOL, max_seq_len=None):
        gpu = self.decode(q, max_seq_len)
        mir = self.mirror.decode(q, self.tinv, self.sm_scale)
        e_m = rel_err(gpu, mir)
        e_r = rel_err(gpu, self.ref.decode(q, self.tinv, self.sm_scale)) if self.ref is not None else 0.0
        assert np.all(np.isfinite(gpu))
        assert e_m <= tol, "decode vs oracle on the GPU's cache: %.3e" % e_m
        assert e_r <= tol, "decode vs oracle from raw inputs: %.3e" % e_r
        return gpu, e_m, e_r

    def reference_for(self, out_fn):
        """(error of the GPU output against the end-to-end reference, tie
        positions substituted) where ``out_fn(cache)`` evaluates the oracle's
        attention on a cache: the reference itself when its key codes equal
        the GPU's, else the reference with the GPU's k~ at the positions whose
        codes differ (tie_patched).  The caller asserts the error."""
        same = all(np.array_equal(self.mirror.kc[b], self.ref.kc[b]) for b in range(self.batch))
        if same:
            return out_fn(self.ref), 0
        patched, n = tie_patched(self.ref, self.mirror)
        return out_fn(patched), n
