"""Pins of the oracle's quantiser (Eq. (7)) against what the paper and
arithmetic fix: hand-worked examples, numpy's linear quantile, the code
range, nearest-level brute force, equivariances, clipping bounds and the
kappa = 1 min-max special case."""
import os

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "quantizer_worked_examples.txt")


def _golden():
    rows = []
    for line in open(GOLDEN):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        head, xs, codes, prm = [p.strip() for p in line.split("|")]
        name, d, bits, kappa = head.split()
        rows.append((name, int(d), int(bits), float(kappa),
                     np.array([float(v) for v in xs.split()], np.float32),
                     np.array([int(v) for v in codes.split()], np.uint8),
                     tuple(int(v, 16) for v in prm.split())))
    return rows


@pytest.mark.parametrize("row", _golden(), ids=lambda r: r[0])
def test_worked_examples(row):
    name, d, bits, kappa, x, codes, (s16, z16) = row
    c, s, z = oracle.quantize_groups(x[None, :], bits, kappa)
    assert c[0].tolist() == codes.tolist()
    assert int(s[0]) == s16 and int(z[0]) == z16


def test_constant_group_reconstructs_exactly():
    x = np.full((1, 8), 0.69921875, np.float32)
    c, s, z = oracle.quantize_groups(x, 2, 1.0)
    assert np.array_equal(oracle.dequant(c, s, z), x)


def _groups(n, d, seed, outliers=True):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((n, d)).astype(np.float32)
    if outliers:
        ch = rng.choice(d, size=4, replace=False)
        x[:, ch] *= 10.0
    # inputs of the quantiser are bf16 values
    return oracle.bf16_to_f32(oracle.f32_to_bf16(x))


@pytest.mark.parametrize("kappa", [0.92, 0.96, 0.99, 0.5, 1.0])
@pytest.mark.parametrize("d", [64, 128])
def test_quantile_matches_numpy_linear(kappa, d):
    x = _groups(400, d, 3)
    for g in x:
        ours = oracle.quantile_abs(g, kappa)
        ref = np.quantile(np.abs(g).astype(np.float64), np.float64(np.float32(kappa)),
                          method="linear")
        # three fp32 roundings vs numpy's fp64: within two fp32 ulps
        assert abs(ours - ref) <= 2 * np.spacing(np.float32(ref)), (ours, ref)


def test_kappa_position_closed_form():
    # pos = kappa (d-1); kappa = 0.96, d = 128 -> 121.92 -> (121, 0.92)
    lo, t = oracle.kappa_position(0.96, 128)
    assert lo == 121 and abs(t - 0.92) < 1e-5
    lo, t = oracle.kappa_position(0.92, 128)
    assert lo == 116 and abs(t - 0.84) < 1e-5
    lo, t = oracle.kappa_position(1.0, 64)
    assert lo == 63 and t == 0.0


@pytest.mark.parametrize("bits", [2, 4])
@pytest.mark.parametrize("kappa", [0.92, 0.96, 1.0])
def test_codes_range_and_clipping(bits, kappa):
    d = 128
    x = _groups(2000, d, 4)
    c, s, z = oracle.quantize_groups(x, bits, kappa)
    assert c.max() <= (1 << bits) - 1
    lo, t = oracle.kappa_position(kappa, d)
    for g in range(0, 2000, 7):
        q = oracle.quantile_abs(x[g], kappa)
        over = np.abs(x[g]) > q
        # at most d-1-lo entries exceed the quantile ...
        assert over.sum() <= d - 1 - lo
        # ... and each of them is clipped to an end code
        assert np.all((c[g][over] == 0) | (c[g][over] == (1 << bits) - 1))


@pytest.mark.parametrize("bits", [2, 4])
def test_nearest_level_brute_force(bits):
    d = 16
    x = _groups(3000, d, 5, outliers=False)
    kappa = 0.9
    c, s16, z16 = oracle.quantize_groups(x, bits, kappa)
    s = oracle.f16_to_f32(s16).astype(np.float64)
    z = oracle.f16_to_f32(z16).astype(np.float64)
    levels = np.arange(1 << bits, dtype=np.float64)
    for g in range(x.shape[0]):
        if s[g] == 0:
            assert np.all(c[g] == 0)
            continue
        recon = s[g] * levels + z[g]
        dist = np.abs(x[g][:, None].astype(np.float64) - recon[None, :])
        best = dist.min(axis=1)
        chosen = dist[np.arange(d), c[g]]
        # the chosen level is the nearest one, up to fp32 rounding of the
        # scaled offset near a tie (half a level apart from two levels)
        assert np.all(chosen <= best + 1e-6 * s[g] + 1e-30), (g, c[g])


@pytest.mark.parametrize("bits", [2, 4])
def test_power_of_two_scale_equivariance(bits):
    x = _groups(1000, 128, 6)
    c0, s0, z0 = oracle.quantize_groups(x, bits, 0.96)
    for k in (-3, 1, 4):
        c1, s1, z1 = oracle.quantize_groups(x * np.float32(2.0 ** k), bits, 0.96)
        assert np.array_equal(c0, c1)
        assert np.array_equal(oracle.f16_to_f32(s1), oracle.f16_to_f32(s0) * np.float32(2.0 ** k))


def test_channel_permutation_equivariance():
    x = _groups(500, 128, 7)
    perm = np.random.default_rng(8).permutation(128)
    c0, s0, z0 = oracle.quantize_groups(x, 2, 0.92)
    c1, s1, z1 = oracle.quantize_groups(x[:, perm], 2, 0.92)
    assert np.array_equal(c0[:, perm], c1)
    assert np.array_equal(s0, s1) and np.array_equal(z0, z1)


def test_kappa_one_is_min_max():
    x = _groups(500, 64, 9)
    c, s, z = oracle.quantize_groups(x, 2, 1.0)
    rows = np.arange(x.shape[0])
    assert np.all(c[rows, x.argmin(axis=1)] == 0)
    assert np.all(c[rows, x.argmax(axis=1)] == 3)


def test_reconstruction_error_bound_and_bits_order():
    x = _groups(2000, 128, 10)
    errs = {}
    for bits in (2, 4):
        c, s, z = oracle.quantize_groups(x, bits, 1.0)
        xh = oracle.dequant(c, s, z)
        sf = oracle.f16_to_f32(s)
        # unclipped (kappa = 1): every entry within half a step (plus fp16 slack
        # of the zero point, at most half an fp16 ulp of x_min)
        slack = np.abs(x.min(axis=1)) * 2.0 ** -11
        assert np.all(np.abs(xh - x) <= (0.5 * sf + slack + 1e-6 * sf)[:, None])
        errs[bits] = np.mean((xh - x) ** 2)
    assert errs[4] < errs[2] / 8


def test_python_dequant_matches_c_fma():
    rng = np.random.default_rng(11)
    s16 = oracle.f32_to_f16(np.abs(rng.standard_normal(5000)).astype(np.float32))
    z16 = oracle.f32_to_f16(rng.standard_normal(5000).astype(np.float32) * 3)
    c = rng.integers(0, 16, 5000).astype(np.uint8)
    L = oracle.lib()
    ref = np.array([L.orc_dequant(int(c[i]), int(s16[i]), int(z16[i])) for i in range(5000)],
                   np.float32)
    ours = oracle.dequant(c[:, None], s16, z16)[:, 0]
    assert np.array_equal(ours, ref)
