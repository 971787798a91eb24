"""Pins of the oracle's RoPE(Norm(k)) for new keys (Eq. (2), Alg. 2 step 1;
RMS normalisation and the pairwise rotations as written in the appendix on
RoPE-commuting transforms): hand-derived worked examples, and properties the
definitions fix (rotations preserve pair norms, scores depend only on the
position difference, the normalisation is scale invariant and gives unit
RMS), plus agreement with the input generator's separate float32 path."""
import os

import numpy as np
import pytest

import oracle
from workloads import synth

HERE = os.path.dirname(os.path.abspath(__file__))


def _examples():
    out = []
    for ln in open(os.path.join(HERE, "golden", "norm_rope_worked_examples.txt")):
        ln = ln.strip()
        if not ln or ln.startswith("#"):
            continue
        theta, pos, eps, x, gain, exp = [f.strip() for f in ln.split("|")]
        out.append((float(theta), int(pos), float(eps), [float(v) for v in x.split()],
                    [float(v) for v in gain.split()], [float(v) for v in exp.split()]))
    return out


@pytest.mark.parametrize("ex", _examples())
def test_worked_examples(ex):
    theta, pos, eps, x, gain, exp = ex
    k = oracle.f64_to_bf16(np.array([x], np.float64))
    got = oracle.norm_rope(k, [pos], theta, gain=np.array(gain), eps=eps)
    want = oracle.f64_to_bf16(np.array([exp], np.float64))
    assert np.array_equal(got, want), (oracle.bf16_to_f32(got), exp)


def _keys(seed, n, d, scale=1.0):
    rng = np.random.default_rng(seed)
    return oracle.f32_to_bf16(rng.standard_t(3.0, size=(n, d)).astype(np.float32) * scale)


def test_position_zero_is_unit_rms_normalisation():
    k = _keys(1, 64, 128)
    out = oracle.bf16_to_f32(oracle.norm_rope(k, np.zeros(64, int), 1e6)).astype(np.float64)
    rms = np.sqrt(np.mean(out ** 2, axis=1))
    assert np.all(np.abs(rms - 1.0) < 2 ** -8)


def test_scale_invariance_is_exact_for_powers_of_two():
    k = _keys(2, 32, 128)
    k4 = oracle.f32_to_bf16(oracle.bf16_to_f32(k) * np.float32(4.0))
    pos = np.arange(32) * 37
    assert np.array_equal(oracle.norm_rope(k, pos, 1e6), oracle.norm_rope(k4, pos, 1e6))


def test_rotation_preserves_pair_norms():
    k = _keys(3, 32, 128)
    y0 = oracle.bf16_to_f32(oracle.norm_rope(k, np.zeros(32, int), 1e4)).astype(np.float64)
    y = oracle.bf16_to_f32(oracle.norm_rope(k, np.arange(32) * 1000 + 5, 1e4)).astype(np.float64)
    n0 = np.hypot(y0[:, :64], y0[:, 64:])
    n1 = np.hypot(y[:, :64], y[:, 64:])
    # each side carries at most one bf16 rounding per coordinate
    assert np.all(np.abs(n1 - n0) <= 2 ** -7 * np.maximum(n0, 1e-30) + 1e-30)
    assert not np.array_equal(y, y0)


def test_scores_depend_only_on_position_difference():
    q = _keys(4, 16, 128)
    k = _keys(5, 16, 128)
    m = np.arange(16) * 300 + 1000
    n = np.arange(16) * 7 + 20
    a = oracle.bf16_to_f32(oracle.norm_rope(q, m, 1e6)).astype(np.float64)
    b = oracle.bf16_to_f32(oracle.norm_rope(k, n, 1e6)).astype(np.float64)
    c = oracle.bf16_to_f32(oracle.norm_rope(q, m - n, 1e6)).astype(np.float64)
    e = oracle.bf16_to_f32(oracle.norm_rope(k, np.zeros(16, int), 1e6)).astype(np.float64)
    lhs = np.sum(a * b, axis=1)
    rhs = np.sum(c * e, axis=1)
    # both sides are dot products of unit-RMS vectors (|.| ~ 11.3) rounded
    # to bf16 coordinatewise
    assert np.all(np.abs(lhs - rhs) < 0.05 * np.sqrt(128))


def test_eps_and_gain():
    k = _keys(6, 8, 64)
    g = np.linspace(0.5, 2.0, 64)
    plain = oracle.bf16_to_f32(oracle.norm_rope(k, np.zeros(8, int), 1e4)).astype(np.float64)
    gained = oracle.bf16_to_f32(oracle.norm_rope(k, np.zeros(8, int), 1e4, gain=g)).astype(np.float64)
    assert np.allclose(gained, plain * g, rtol=2 ** -7, atol=1e-6)
    big = oracle.bf16_to_f32(oracle.norm_rope(k, np.zeros(8, int), 1e4, eps=1e12)).astype(np.float64)
    assert np.all(np.abs(big) < 1e-3)


def test_agrees_with_generator_float32_path():
    """The workload generator's own RMS normalisation and rotation (float32,
    written separately for the inputs) lands within one bf16 step of the
    oracle on the same bf16 pre-normalisation keys."""
    w = synth.Workload(synth.CONFIGS["prefill"])
    raw = w.raw_keys(0, 100, 64)                              # [64][n_kv][d]
    x = oracle.bf16_to_f32(raw).astype(np.float64)
    rms = np.sqrt(np.mean(x ** 2, axis=-1, keepdims=True))
    gen = synth.to_bf16_bits(synth.rope((x / rms).astype(np.float32), np.arange(100, 164), 1e6))
    ours = oracle.norm_rope(np.transpose(raw, (1, 0, 2)), np.arange(100, 164), 1e6)
    ours = np.transpose(ours, (1, 0, 2))
    a = oracle.bf16_to_f32(gen).astype(np.float64)
    b = oracle.bf16_to_f32(ours).astype(np.float64)
    step = np.abs(b) * 2 ** -7 + 1e-30
    assert np.all(np.abs(a - b) <= 1.01 * step)
    assert np.mean(a != b) < 0.05
