"""Pins of the oracle's QuEST quantiser (Eq. (5), Sec. 4.3) and of its clip
multiplier alpha_b against what the paper and the mathematics fix: worked
examples, the one-bit closed form, the stationarity identity and the clipping
bound of the Gaussian-clipping lemma (App. B), a direct quadrature of the
error, the nearest-level property of the reconstruction, equivariances, and
the Gaussian error the grid must reach."""
import math
import os

import numpy as np
import pytest
from scipy import integrate

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "quest_worked_examples.txt")


def _golden():
    rows = []
    for line in open(GOLDEN):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        head, xs, codes, prm = [p.strip() for p in line.split("|")]
        name, d, bits, alpha = head.split()
        rows.append((name, int(d), int(bits), float(alpha),
                     np.array([float(v) for v in xs.split()], np.float32),
                     np.array([int(v) for v in codes.split()], np.uint8),
                     tuple(int(v, 16) for v in prm.split())))
    return rows


@pytest.mark.parametrize("row", _golden(), ids=lambda r: r[0])
def test_worked_examples(row):
    name, d, bits, alpha, x, codes, (s16, z16) = row
    assert x.size == d
    c, s, z = oracle.quest_quantize_groups(x[None, :], bits, alpha)
    assert c[0].tolist() == codes.tolist()
    assert int(s[0]) == s16 and int(z[0]) == z16


# ---------------------------------------------------------------- alpha_b

def _nearest_level(t, alpha, bits):
    n = 1 << bits
    lv = -alpha + 2.0 * alpha / (n - 1) * np.arange(n)
    return lv[np.argmin(np.abs(lv[None, :] - np.atleast_1d(t)[:, None]), axis=1)]


def _quad_moments(alpha, bits):
    """E[zh^2], E[z zh], E[(zh - z)^2] and E[(|z| - alpha)_+^2] for z standard
    Gaussian and zh its nearest level, by adaptive quadrature over each cell
    (independent of the closed-form error the oracle minimises)."""
    n = 1 << bits
    lv = -alpha + 2.0 * alpha / (n - 1) * np.arange(n)
    edges = [-np.inf] + list(0.5 * (lv[1:] + lv[:-1])) + [np.inf]
    phi = lambda t: math.exp(-0.5 * t * t) / math.sqrt(2.0 * math.pi)
    m_hh = m_zh = mse = 0.0
    for k in range(n):
        a, b, l = edges[k], edges[k + 1], lv[k]
        m_hh += l * l * integrate.quad(phi, a, b, epsabs=1e-14, epsrel=1e-13)[0]
        m_zh += l * integrate.quad(lambda t: t * phi(t), a, b, epsabs=1e-14, epsrel=1e-13)[0]
        mse += integrate.quad(lambda t: (t - l) ** 2 * phi(t), a, b, epsabs=1e-14, epsrel=1e-13)[0]
    clip = 2.0 * integrate.quad(lambda t: (t - alpha) ** 2 * phi(t), alpha, np.inf,
                                epsabs=1e-15, epsrel=1e-13)[0]
    return m_hh, m_zh, mse, clip


def test_alpha_one_bit_closed_form():
    # two levels +-alpha: error 1 - 2 alpha E|z| + alpha^2, least at E|z| = sqrt(2/pi)
    assert abs(oracle.quest_alpha(1) - math.sqrt(2.0 / math.pi)) < 1e-6


@pytest.mark.parametrize("bits", [1, 2, 3, 4, 5, 6])
def test_alpha_stationarity_and_clip_bound(bits):
    """App. B, Gaussian-clipping lemma: at the optimal endpoint the second
    moment of the reconstruction equals its correlation with the input, and
    the clipping error is at most (2^b - 1)^-2."""
    a = oracle.quest_alpha(bits)
    m_hh, m_zh, mse, clip = _quad_moments(a, bits)
    assert abs(m_hh - m_zh) < 1e-6
    assert clip <= (2 ** bits - 1) ** -2
    # the closed-form error the oracle minimises equals the quadrature
    assert abs(oracle.quest_grid_mse(a, bits) - mse) < 1e-10
    # and alpha_b is a minimum: moving it either way costs error
    for f in (0.99, 1.01):
        assert _quad_moments(a * f, bits)[2] > mse


def test_alpha_grows_with_bits():
    al = [oracle.quest_alpha(b) for b in range(1, 9)]
    assert all(b > a for a, b in zip(al, al[1:]))


def test_alpha_textbook_steps():
    # Max (1960), optimum uniform quantiser of a unit Gaussian: steps 0.9957,
    # 0.5860, 0.3352 for 4, 8 and 16 levels (step = 2 alpha_b / (2^b - 1))
    for bits, step in ((2, 0.9957), (3, 0.5860), (4, 0.3352)):
        assert abs(2.0 * oracle.quest_alpha(bits) / (2 ** bits - 1) - step) < 1e-4


# ---------------------------------------------------------------- quantiser

def _groups(seed, n, d, scale=1.0):
    rng = np.random.default_rng(seed)
    x = (rng.standard_normal((n, d)) * scale).astype(np.float32)
    x[:, rng.integers(0, d, 3)] *= 8.0  # a few outlier channels
    return x


@pytest.mark.parametrize("bits", [2, 4])
def test_codes_in_range_and_zero_group(bits):
    x = _groups(1, 200, 128)
    x[7] = 0.0
    c, s, z = oracle.quest_quantize_groups(x, bits, oracle.quest_alpha(bits))
    assert c.max() <= 2 ** bits - 1
    assert np.all(oracle.dequant(c[7], s[7], z[7]) == 0.0)


@pytest.mark.parametrize("bits", [2, 4])
def test_reconstruction_is_nearest_level(bits):
    """Every reconstruction is the level of the stored grid nearest to x, the
    grid being the 2^b bin centres; clipped entries take an end level."""
    alpha = oracle.quest_alpha(bits)
    x = _groups(2, 300, 64)
    c, s16, z16 = oracle.quest_quantize_groups(x, bits, alpha)
    xh = oracle.dequant(c, s16, z16).astype(np.float64)
    s = oracle.f16_to_f32(s16).astype(np.float64)
    lv = (s[:, None] * (np.arange(2 ** bits)[None, :] + 0.5 - 2 ** (bits - 1)))  # [n][levels]
    y = x / s[:, None]
    away = np.abs(y - np.round(y)) > 1e-3  # not within rounding of a cell edge
    for g in range(x.shape[0]):
        near = lv[g][np.argmin(np.abs(lv[g][None, :] - x[g][:, None].astype(np.float64)), axis=1)]
        # the stored zero is fp16-rounded: levels agree to 2^-11 of the zero
        tol = 2.0 ** -11 * abs(float(oracle.f16_to_f32(z16[g]))) + 1e-12
        assert np.all(np.abs(xh[g] - near)[away[g]] <= tol)


@pytest.mark.parametrize("bits", [2, 4])
def test_levels_span_alpha_rms(bits):
    alpha = oracle.quest_alpha(bits)
    x = _groups(3, 50, 128)
    c, s16, z16 = oracle.quest_quantize_groups(x, bits, alpha)
    top = oracle.dequant(np.full((50, 1), 2 ** bits - 1, np.uint8), s16, z16)[:, 0]
    bot = oracle.dequant(np.zeros((50, 1), np.uint8), s16, z16)[:, 0]
    rms = np.sqrt(np.mean(x.astype(np.float64) ** 2, axis=1))
    assert np.allclose(top, alpha * rms, rtol=2e-3)
    assert np.allclose(bot, -alpha * rms, rtol=2e-3)


@pytest.mark.parametrize("bits", [2, 4])
def test_power_of_two_equivariance_and_antisymmetry(bits):
    alpha = oracle.quest_alpha(bits)
    x = _groups(4, 100, 128)
    c, s, z = oracle.quest_quantize_groups(x, bits, alpha)
    c4, s4, z4 = oracle.quest_quantize_groups(4.0 * x, bits, alpha)
    assert np.array_equal(c, c4)
    assert np.array_equal(oracle.f16_to_f32(s4), 4.0 * oracle.f16_to_f32(s))
    assert np.array_equal(oracle.f16_to_f32(z4), 4.0 * oracle.f16_to_f32(z))
    cn, sn, zn = oracle.quest_quantize_groups(-x, bits, alpha)
    assert np.array_equal(s, sn)
    inv = 1.0 / oracle.f16_to_f32(s)
    y = x * inv[:, None]
    inner = y != np.floor(y)  # off the cell edges, floor(-y) = -floor(y) - 1
    assert np.array_equal(cn[inner], (2 ** bits - 1 - c.astype(int))[inner])


@pytest.mark.parametrize("bits", [2, 3, 4])
def test_gaussian_error_matches_the_grid(bits):
    """Wide Gaussian groups (RMS within a percent of 1): the relative error of
    the RMS-scaled grid is the fixed grid's Gaussian error at alpha_b."""
    alpha = oracle.quest_alpha(bits)
    x = np.random.default_rng(5).standard_normal((64, 8192)).astype(np.float32)
    c, s, z = oracle.quest_quantize_groups(x, bits, alpha)
    err = np.mean((oracle.dequant(c, s, z).astype(np.float64) - x) ** 2)
    ref = oracle.quest_grid_mse(alpha, bits)
    assert abs(err / np.mean(x.astype(np.float64) ** 2) - ref) < 0.02 * ref


def test_cache_flush_time_independence_quest():
    """A QuEST cache filled by one append equals one filled token by token."""
    rng = np.random.default_rng(6)
    d, H, S = 64, 2, 300
    alpha = oracle.quest_alpha(2)
    k = oracle.f32_to_bf16(rng.standard_normal((1, S, H, d)).astype(np.float32))
    v = oracle.f32_to_bf16(rng.standard_normal((1, S, H, d)).astype(np.float32))
    tk = oracle.f32_to_bf16(np.broadcast_to(np.eye(d, dtype=np.float32), (H, d, d)).copy())
    args = (1, H, d, 2, 4, 32, 8, 0.96, 0.92, 512)
    a = oracle.OracleCache(*args, codec="quest", quest_alpha=alpha)
    a.append(k, v, [S], tk)
    b = oracle.OracleCache(*args, codec="quest", quest_alpha=alpha)
    for t in range(S):
        b.append(k[:, t:t + 1], v[:, t:t + 1], [1], tk)
    for name in ("kc", "vc", "kp", "vp", "seq_len", "quant_end"):
        assert np.array_equal(getattr(a, name), getattr(b, name)), name
    # and it is not the percentile codec
    p = oracle.OracleCache(*args)
    p.append(k, v, [S], tk)
    assert not np.array_equal(a.kc, p.kc)
