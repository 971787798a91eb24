"""Seeded synthetic workloads.

The paper's inputs are Qwen3 / Llama activations on text corpora that are not
available here; these generators stand in for them with the shapes and value
structure the workloads call for:

  keys    post-RoPE Gaussian with a few seeded outlier channels scaled up
          (a common structure of real key caches), or heavy-tailed Student-t
          (nu = 3) followed by headwise RMS normalisation and RoPE;
  values  standard Gaussian (already in transformed coordinates);
  queries standard Gaussian, RoPE'd at the decode position;
  T_K     Q diag(s) Q^T per kv head with Q Haar-orthogonal and s log-uniform
          in [0.5, 2] (or Q1 diag(s) Q2^T, which is not symmetric).

Every draw comes from numpy's PCG64 seeded with (seed, tag), so a tensor is
reproducible by itself.  bf16 rounding of generated floats uses torch's cast.
"""
from __future__ import annotations

import dataclasses
import zlib

import numpy as np

CONFIGS = {
    # tiny parity case
    "tiny": dict(batch=1, n_kv=1, n_q=4, d=64, ctx=512, bits=2, s_sink=4, s_keep=32,
                 s_flush=8, kappa_k=0.99, kappa_v=0.99, k_dist="gauss", outliers=4,
                 outlier_scale=8.0, v_outliers=True, rope_theta=None),
    # Llama-3-8B-shaped decode layer
    "llama8b": dict(batch=8, n_kv=8, n_q=32, d=128, ctx=8192, bits=2, s_sink=4, s_keep=128,
                    s_flush=8, kappa_k=0.96, kappa_v=0.92, k_dist="gauss", outliers=8,
                    outlier_scale=10.0, v_outliers=False, rope_theta=5.0e5),
    # Qwen3-32B-shaped decode layer: 64 query heads on 8 kv heads (eight per
    # kv head), same cache recipe as the Llama-shaped one
    "qwen32b": dict(batch=8, n_kv=8, n_q=64, d=128, ctx=8192, bits=2, s_sink=4, s_keep=128,
                    s_flush=8, kappa_k=0.96, kappa_v=0.92, k_dist="gauss", outliers=8,
                    outlier_scale=10.0, v_outliers=False, rope_theta=1.0e6),
    # long context, paged in random physical order
    "long2": dict(batch=1, n_kv=8, n_q=32, d=128, ctx=131072, bits=2, s_sink=4, s_keep=128,
                  s_flush=8, kappa_k=0.96, kappa_v=0.92, k_dist="gauss", outliers=8,
                  outlier_scale=10.0, v_outliers=False, rope_theta=5.0e5,
                  page_order="random", pool_factor=1.25),
    "long4": dict(batch=1, n_kv=8, n_q=32, d=128, ctx=131072, bits=4, s_sink=4, s_keep=128,
                  s_flush=8, kappa_k=0.96, kappa_v=0.92, k_dist="gauss", outliers=8,
                  outlier_scale=10.0, v_outliers=False, rope_theta=5.0e5,
                  page_order="random", pool_factor=1.25),
    # large batch, ragged lengths
    "bigbatch": dict(batch=64, n_kv=8, n_q=32, d=128, ctx=32768, ctx_min=16384, bits=2,
                     s_sink=4, s_keep=128, s_flush=8, kappa_k=0.96, kappa_v=0.92,
                     k_dist="gauss", outliers=8, outlier_scale=10.0, v_outliers=False,
                     rope_theta=5.0e5),
    # prefill append: 4 x 16384 new tokens, QK-norm + RoPE (theta 1e6)
    "prefill": dict(batch=4, n_kv=8, n_q=64, d=128, ctx=16384, bits=2, s_sink=4, s_keep=128,
                    s_flush=8, kappa_k=0.96, kappa_v=0.92, k_dist="student_t3_rmsnorm",
                    outliers=0, outlier_scale=1.0, v_outliers=False, rope_theta=1.0e6),
}


def make_rng(seed: int, tag: str) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, zlib.crc32(tag.encode())])))


def random_orthogonal(d: int, rng: np.random.Generator) -> np.ndarray:
    """Haar-distributed orthogonal matrix: QR of a Gaussian, signs fixed by R's diagonal."""
    a = rng.standard_normal((d, d))
    q, r = np.linalg.qr(a)
    return q * np.sign(np.diag(r))[None, :]


def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """float array -> bf16 bit patterns (uint16) via torch's round-to-nearest-even cast."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16).copy()


def bf16_bits_to_float(h: np.ndarray) -> np.ndarray:
    return (np.asarray(h, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def make_transform(n_kv: int, d: int, seed: int = 0, symmetric: bool = True, tag: str = "tk"):
    """Per-head T_K as bf16 bits [n_kv][d][d] and its inverse (fp64 inverse of
    the bf16-rounded matrix, stored as fp32)."""
    rng = make_rng(seed, tag)
    tk = np.empty((n_kv, d, d), np.float64)
    for h in range(n_kv):
        q1 = random_orthogonal(d, rng)
        q2 = q1 if symmetric else random_orthogonal(d, rng)
        s = np.exp(rng.uniform(np.log(0.5), np.log(2.0), size=d))
        tk[h] = (q1 * s[None, :]) @ q2.T
    tk_bits = to_bf16_bits(tk)
    tk_b = bf16_bits_to_float(tk_bits).astype(np.float64)
    tinv = np.stack([np.linalg.inv(tk_b[h]) for h in range(n_kv)]).astype(np.float32)
    return tk_bits, tinv


@dataclasses.dataclass
class Workload:
    """Inputs of one configuration: per-sequence keys / values as bf16 bits
    [batch][n][n_kv][d] (row t = position t), lengths, queries, transforms."""
    cfg: dict
    seed: int = 0
    symmetric_tk: bool = True

    def __post_init__(self):
        c = self.cfg
        self.batch, self.n_kv, self.n_q, self.d = c["batch"], c["n_kv"], c["n_q"], c["d"]
        self.G = self.n_q // self.n_kv
        rng = make_rng(self.seed, "lengths")
        if "ctx_min" in c:
            self.lengths = rng.integers(c["ctx_min"], c["ctx"] + 1, size=self.batch).astype(np.int32)
        else:
            self.lengths = np.full(self.batch, c["ctx"], np.int32)
        ch_rng = make_rng(self.seed, "outlier_channels")
        self.k_outlier_ch = np.sort(ch_rng.choice(self.d, size=c["outliers"], replace=False)) \
            if c["outliers"] else np.zeros(0, np.int64)
        self.v_outlier_ch = np.sort(ch_rng.choice(self.d, size=c["outliers"], replace=False)) \
            if (c["outliers"] and c["v_outliers"]) else np.zeros(0, np.int64)

    def transform(self):
        return make_transform(self.n_kv, self.d, self.seed, self.symmetric_tk)

    def keys(self, b: int, start: int, n: int) -> np.ndarray:
        """bf16 bits [n][n_kv][d] of sequence b, positions start .. start+n-1."""
        c = self.cfg
        rng = make_rng(self.seed * 1000003 + b, "keys@%d" % start)
        if c["k_dist"] == "gauss":
            x = rng.standard_normal((n, self.n_kv, self.d), dtype=np.float32)
            if len(self.k_outlier_ch):
                x[..., self.k_outlier_ch] *= np.float32(c["outlier_scale"])
        elif c["k_dist"] == "student_t3_rmsnorm":
            x = rng.standard_t(3.0, size=(n, self.n_kv, self.d)).astype(np.float32)
            rms = np.sqrt(np.mean(x.astype(np.float64) ** 2, axis=-1, keepdims=True))
            x = (x / rms).astype(np.float32)
        else:
            raise ValueError(c["k_dist"])
        if c["rope_theta"]:
            pos = np.arange(start, start + n)
            x = rope(x, pos, c["rope_theta"])
        return to_bf16_bits(x)

    def raw_keys(self, b: int, start: int, n: int) -> np.ndarray:
        """bf16 bits [n][n_kv][d] of keys before headwise normalisation and
        RoPE (the input of the fused norm + RoPE append): the Student-t or
        Gaussian draw of keys() without its normalisation and rotation."""
        c = self.cfg
        rng = make_rng(self.seed * 1000003 + b, "raw_keys@%d" % start)
        if c["k_dist"] == "gauss":
            x = rng.standard_normal((n, self.n_kv, self.d), dtype=np.float32)
            if len(self.k_outlier_ch):
                x[..., self.k_outlier_ch] *= np.float32(c["outlier_scale"])
        elif c["k_dist"] == "student_t3_rmsnorm":
            x = rng.standard_t(3.0, size=(n, self.n_kv, self.d)).astype(np.float32)
        else:
            raise ValueError(c["k_dist"])
        return to_bf16_bits(x)

    def values(self, b: int, start: int, n: int) -> np.ndarray:
        c = self.cfg
        rng = make_rng(self.seed * 1000003 + b, "values@%d" % start)
        x = rng.standard_normal((n, self.n_kv, self.d), dtype=np.float32)
        if len(self.v_outlier_ch):
            x[..., self.v_outlier_ch] *= np.float32(c["outlier_scale"])
        return to_bf16_bits(x)

    def query(self, step: int = 0) -> np.ndarray:
        """bf16 bits [batch][n_q][d] of the decode query at position len - 1 (+ step)."""
        c = self.cfg
        rng = make_rng(self.seed, "query@%d" % step)
        x = rng.standard_normal((self.batch, self.n_q, self.d), dtype=np.float32)
        if c["rope_theta"]:
            out = np.empty_like(x)
            for b in range(self.batch):
                pos = np.array([self.lengths[b] - 1 + step])
                out[b] = rope(x[b][None], pos, c["rope_theta"])[0]
            x = out
        return to_bf16_bits(x)


def rope_table(theta: float, d: int, max_pos: int) -> np.ndarray:
    """The model's rotary table, fp32 [max_pos][d]: cos(s w_j) in columns
    j < d/2 and sin(s w_j) in columns d/2 + j, w_j = theta^(-2j/d), evaluated
    in fp64 and rounded once."""
    half = d // 2
    w = float(theta) ** (-np.arange(half, dtype=np.float64) * 2.0 / d)
    ang = np.arange(max_pos, dtype=np.float64)[:, None] * w[None, :]
    return np.concatenate([np.cos(ang), np.sin(ang)], axis=1).astype(np.float32)


def rope(x: np.ndarray, positions: np.ndarray, theta: float) -> np.ndarray:
    """Rotate-half RoPE for x [S][heads][d] at the given S positions."""
    d = x.shape[-1]
    half = d // 2
    inv = theta ** (-np.arange(half, dtype=np.float64) * 2.0 / d)
    ang = positions.astype(np.float64)[:, None] * inv[None, :]
    cos = np.cos(ang)[:, None, :].astype(np.float32)
    sin = np.sin(ang)[:, None, :].astype(np.float32)
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * cos - x2 * sin, x2 * cos + x1 * sin], axis=-1)
