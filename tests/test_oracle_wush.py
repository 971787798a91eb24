"""Pins of the oracle's WUSH transform (Eq. (1), Sec. 3) against what the
paper proves about it: Frobenius-norm preservation at gamma = 0, invariance to
rescaling either statistic, the equalisation identity and sensitivity balance
(App. B, Theorem on the unclipped optimum), attainment of that theorem's
lower bound (computed from an independent SVD of M^1/2 H^1/2) while other
transforms stay above it, and the diagonal case."""
import numpy as np
import pytest
from scipy import linalg as sla

import oracle


def _stats(seed, d, n_m=400, n_h=300, outliers=4):
    rng = np.random.default_rng(seed)
    X = rng.standard_normal((d, n_m))
    X[rng.choice(d, outliers, replace=False)] *= 8.0
    Q = rng.standard_normal((d, n_h)) * rng.uniform(0.3, 3.0, (d, 1))
    return X, X @ X.T, 2.0 * Q @ Q.T


def test_hadamard_is_orthogonal_sylvester():
    for d in (2, 8, 64, 128):
        Hd = oracle.sylvester_hadamard(d)
        assert np.allclose(Hd @ Hd.T, np.eye(d), atol=1e-12)
        assert np.allclose(np.abs(Hd), d ** -0.5)
        assert np.allclose(Hd, sla.hadamard(d) / np.sqrt(d))  # Sylvester's order
    h2 = oracle.sylvester_hadamard(2) * np.sqrt(2)
    assert np.array_equal(h2, [[1, 1], [1, -1]])


@pytest.mark.parametrize("d", [16, 64, 128])
def test_frobenius_norm_preserved_undamped(d):
    X, M, H = _stats(d, d)
    T, Ti, _ = oracle.wush_transform(M, H, 0.0)
    assert abs(np.linalg.norm(T @ X) / np.linalg.norm(X) - 1.0) < 1e-10
    assert np.allclose(T @ Ti, np.eye(d), atol=1e-9)


@pytest.mark.parametrize("gamma", [0.0, 1e-2])
def test_invariant_to_rescaling_the_statistics(gamma):
    _, M, H = _stats(1, 64)
    T, _, _ = oracle.wush_transform(M, H, gamma)
    for rm, rh in ((3.0, 1.0), (1.0, 0.01), (250.0, 7.0)):
        T2, _, _ = oracle.wush_transform(rm * M, rh * H, gamma)
        assert np.allclose(T2, T, rtol=1e-8, atol=1e-10 * np.abs(T).max())


@pytest.mark.parametrize("d", [32, 128])
def test_bound_attained_and_equalised(d):
    """Theorem (App. B): tr(T M T^T) tr(T^-T H T^-1) >= (sum sigma_i)^2 for
    every invertible T, sigma the singular values of M^1/2 H^1/2; the
    undamped WUSH transform attains it, with both products proportional
    (equalisation) and their diagonals constant (sensitivity balance)."""
    _, M, H = _stats(2 + d, d)
    sig = np.linalg.svd(np.real(sla.sqrtm(M)) @ np.real(sla.sqrtm(H)), compute_uv=False)
    bound = np.sum(sig) ** 2
    T, Ti, _ = oracle.wush_transform(M, H, 0.0)
    A = T @ M @ T.T
    B = Ti.T @ H @ Ti
    assert abs(np.trace(A) * np.trace(B) / bound - 1.0) < 1e-8
    ratio = np.trace(A) / np.trace(B)
    assert np.allclose(A, ratio * B, rtol=1e-7, atol=1e-9 * np.abs(A).max())
    assert np.allclose(np.diag(A), np.trace(A) / d, rtol=1e-8)
    assert np.allclose(np.diag(B), np.trace(B) / d, rtol=1e-8)
    rng = np.random.default_rng(d)
    for _ in range(5):  # other transforms stay above the bound
        T2 = rng.standard_normal((d, d)) + 3 * np.eye(d)
        T2i = np.linalg.inv(T2)
        assert np.trace(T2 @ M @ T2.T) * np.trace(T2i.T @ H @ T2i) > bound * (1 + 1e-6)
    Qo, _ = np.linalg.qr(rng.standard_normal((d, d)))  # orthogonal: tr(M) tr(H)
    assert abs(np.trace(Qo @ M @ Qo.T) * np.trace(Qo @ H @ Qo.T) / (np.trace(M) * np.trace(H)) - 1) < 1e-10


def test_damped_products_stay_equalised():
    """With damping the same identities hold for the damped statistics, and
    the norm grows by exactly (1 + gamma)."""
    d, g = 64, 1e-2
    _, M, H = _stats(5, d)
    T, Ti, _ = oracle.wush_transform(M, H, g)
    Md = M + g * np.trace(M) / d * np.eye(d)
    Hd = H + g * np.trace(H) / d * np.eye(d)
    A = T @ Md @ T.T
    B = Ti.T @ Hd @ Ti
    assert abs(np.trace(A) / ((1 + g) * np.trace(M)) - 1) < 1e-10
    assert np.allclose(np.diag(A), np.trace(A) / d, rtol=1e-8)
    assert np.allclose(A, np.trace(A) / np.trace(B) * B, rtol=1e-7, atol=1e-9 * np.abs(A).max())


def test_diagonal_statistics():
    """M = diag(m), H = diag(h): L = diag(sqrt h), the eigenvalues are h m
    in ascending order with unit eigenvectors, so row i of T is c times the
    Hadamard row i spread over the sorted coordinates, each scaled by
    (h m)^(-1/4) sqrt(h)."""
    rng = np.random.default_rng(6)
    d = 16
    m = rng.uniform(0.5, 4.0, d)
    h = rng.uniform(0.5, 4.0, d)
    T, _, lam = oracle.wush_transform(np.diag(m), np.diag(h), 0.0)
    order = np.argsort(h * m)
    assert np.allclose(lam, (h * m)[order])
    c = np.sqrt(np.sum(m)) / np.sqrt(np.sum(np.sqrt(h * m)))
    want = np.zeros((d, d))
    Hd = sla.hadamard(d) / np.sqrt(d)
    for r, k in enumerate(order):
        want[:, k] = c * Hd[:, r] * (h[k] * m[k]) ** -0.25 * np.sqrt(h[k])
    assert np.allclose(T, want, rtol=1e-10, atol=1e-12)
