"""GPU parity of the WUSH transform builder (Eq. (1)) through the C ABI: T and
T^{-1} against the oracle's fp64 construction from the same fp32 statistics,
plus the identities the paper proves, evaluated on the GPU's own output."""
import numpy as np
import pytest
import torch

from gpu_harness import say
import oracle
import paper_2609_38121_amd as wk
from workloads import synth

pytestmark = pytest.mark.gpu


def _pairs(seed, count, d, gamma=None):
    """Synthetic calibration statistics of the paper's form (Eq. (4)):
    M = K K^T of keys with outlier channels, H = 2 sum_g Q Q^T of the
    group's queries; fp32, exactly symmetric.  With gamma, draws whose
    eigenpairs come within a near-tie of the order or sign rule (where two
    correct constructions differ) are skipped, so that T is comparable
    element by element."""
    rng = np.random.default_rng(seed)
    Ms, Hs, Xs = [], [], []
    while len(Ms) < count:
        n = 512
        K = rng.standard_normal((d, n))
        K[rng.choice(d, 4, replace=False)] *= 10.0
        Q = rng.standard_normal((d, 4 * n)) * rng.uniform(0.3, 3.0, (d, 1))
        M = (K @ K.T / n).astype(np.float32)
        H = (2.0 * Q @ Q.T / n).astype(np.float32)
        M = np.tril(M) + np.tril(M, -1).T
        H = np.tril(H) + np.tril(H, -1).T
        if gamma is not None:
            gap, sign_margin = _margins(M.astype(np.float64), H.astype(np.float64), gamma)
            if gap < 1e-4 or sign_margin < 3e-3:
                continue
        Ms.append(M)
        Hs.append(H)
        Xs.append(K / np.sqrt(n))
    return np.stack(Ms), np.stack(Hs), Xs


def _margins(M, H, gamma):
    """Smallest relative eigenvalue gap and smallest ratio between the two
    largest magnitudes of a column of L U (the sign rule's margin)."""
    d = M.shape[0]
    L = np.linalg.cholesky(H + gamma * np.trace(H) / d * np.eye(d))
    lam, U = np.linalg.eigh(L.T @ (M + gamma * np.trace(M) / d * np.eye(d)) @ L)
    gap = np.min(np.diff(lam) / lam[1:])
    W = np.sort(np.abs(L @ U), axis=0)
    return gap, np.min(1.0 - W[-2] / W[-1])


@pytest.mark.parametrize("d,gamma", [(128, 1e-2), (128, 0.0), (64, 1e-2), (64, 0.0)])
def test_wush_transform_matches_oracle(gpu, d, gamma):
    count = 6
    M, H, Xs = _pairs(10 + d + int(gamma * 100), count, d, gamma)
    say("wush d=%d gamma=%g count=%d" % (d, gamma, count))
    T, Ti, sw = wk.wushkv_wush_transform(torch.from_numpy(M).to(gpu), torch.from_numpy(H).to(gpu),
                                         gamma=gamma)
    torch.cuda.synchronize()
    T, Ti, sw = T.cpu().numpy().astype(np.float64), Ti.cpu().numpy().astype(np.float64), sw.cpu().numpy()
    say("  sweeps", sw.tolist())
    assert np.all((sw > 0) & (sw < 40))
    for k in range(count):
        m, h = M[k].astype(np.float64), H[k].astype(np.float64)
        Tr, Tir, _ = oracle.wush_transform(m, h, gamma)
        eT = np.linalg.norm(T[k] - Tr) / np.linalg.norm(Tr)
        eTi = np.linalg.norm(Ti[k] - Tir) / np.linalg.norm(Tir)
        say("  pair %d: |T - T_ref|/|T_ref| %.2e, inverse %.2e" % (k, eT, eTi))
        assert eT < 2e-3 and eTi < 2e-3
        # the paper's identities on the GPU's own T
        assert np.abs(T[k] @ Ti[k] - np.eye(d)).max() < 2e-3
        Md = m + gamma * np.trace(m) / d * np.eye(d)
        A = T[k] @ Md @ T[k].T
        assert abs(np.trace(A) / ((1 + gamma) * np.trace(m)) - 1) < 1e-3
        assert np.allclose(np.diag(A), np.trace(A) / d, rtol=2e-3)
        if gamma == 0.0:
            assert abs(np.linalg.norm(T[k] @ Xs[k]) / np.linalg.norm(Xs[k]) - 1) < 1e-3


def test_wush_transform_not_positive_definite(gpu):
    d = 64
    M, H, _ = _pairs(3, 2, d)
    H[1] = 0.0  # undamped zero Hessian: no Cholesky factor
    T, Ti, sw = wk.wushkv_wush_transform(torch.from_numpy(M).to(gpu), torch.from_numpy(H).to(gpu),
                                         gamma=0.0)
    torch.cuda.synchronize()
    sw = sw.cpu().numpy()
    assert sw[0] > 0 and sw[1] == -1
    assert np.all(np.isfinite(T[0].cpu().numpy())) and np.all(np.isnan(T[1].cpu().numpy()))
    assert np.all(np.isnan(Ti[1].cpu().numpy()))


def test_wush_transform_drives_the_cache(gpu):
    """The built T (as bf16) and T^{-1} run through append and decode, and
    the oracle fed the same transform agrees."""
    from gpu_harness import Pair, rel_err, to_dev_bf16
    d, H_, G = 128, 2, 4
    M, Hm, _ = _pairs(4, H_, d)
    T, Ti, _ = wk.wushkv_wush_transform(torch.from_numpy(M).to(gpu), torch.from_numpy(Hm).to(gpu),
                                        gamma=1e-2)
    tk_bits = oracle.f32_to_bf16(T.cpu().numpy())
    p = Pair(gpu, 2, H_, G, d, 2, 4, 64, 8, 0.96, 0.92, cap=700)
    p.tk, p.tk_dev = tk_bits, to_dev_bf16(tk_bits, gpu)
    # T^{-1} of the bf16 T, in fp64 as the oracle would have it
    p.tinv = np.linalg.inv(oracle.bf16_to_f32(tk_bits).astype(np.float64)).astype(np.float32)
    p.tinv_dev = torch.from_numpy(p.tinv).to(gpu)
    rng = np.random.default_rng(5)
    k = oracle.f32_to_bf16(rng.standard_normal((2, 600, H_, d)).astype(np.float32))
    v = oracle.f32_to_bf16(rng.standard_normal((2, 600, H_, d)).astype(np.float32))
    p.append(k, v, [600, 333])
    assert p.check_cache() > 0
    q = oracle.f32_to_bf16(rng.standard_normal((2, H_ * G, d)).astype(np.float32))
    _, em, er = p.decode_check(q)
    say("  built transform through the cache: rel err %.2e / %.2e" % (em, er))
