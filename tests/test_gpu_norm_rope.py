"""GPU parity of the fused append (headwise RMS normalisation and RoPE of the
new keys in front of the key transform, Alg. 2 step 1) against the oracle.

The mirror oracle cache is fed the GPU's own k~, so codes, parameters and
windows must match bit for bit.  The reference oracle cache is fed
RoPE(Norm(k)) evaluated by the oracle in fp64 and rounded to bf16; the GPU
evaluates it in fp32 and may land on the other bf16 neighbour in rare
elements, so k~ is checked against the fp64 product within the fp32 bound on
all but a small fraction of elements, and decode outputs against both caches
(where a key code of the reference sits on the other side of such a rounding
tie, the reference takes the GPU's k~ at exactly those positions:
gpu_harness.tie_patched)."""
import numpy as np
import pytest

from gpu_harness import Pair, rel_err, say, TOL
import oracle

pytestmark = pytest.mark.gpu


def _raw(rng, B, n, H, d):
    k = rng.standard_t(3.0, size=(B, n, H, d)).astype(np.float32) * 3.0
    v = rng.standard_normal((B, n, H, d)).astype(np.float32)
    return oracle.f32_to_bf16(k), oracle.f32_to_bf16(v)


def _q(rng, B, nq, d):
    return oracle.f32_to_bf16(rng.standard_normal((B, nq, d)).astype(np.float32))


def _check_k_tilde(p, frac=1e-3):
    total, diff, bad = p.k_tilde_vs_ref()
    say("  k~ vs fp64 of the oracle's RoPE(Norm(k)): %d of %d differ, %d outside the bound"
        % (diff, total, bad))
    assert bad <= frac * total


def _decode(p, q):
    gpu = p.decode(q)
    mir = p.mirror.decode(q, p.tinv, p.sm_scale)
    ref, n_sub = p.reference_for(lambda c: c.decode(q, p.tinv, p.sm_scale))
    em, er = rel_err(gpu, mir), rel_err(gpu, ref)
    say("  decode rel err vs mirror %.2e, vs reference %.2e (%d tie positions substituted)"
        % (em, er, n_sub))
    assert np.all(np.isfinite(gpu))
    assert em <= TOL
    assert er <= TOL


@pytest.mark.parametrize("d,bits,G,use_gain", [(128, 2, 4, True), (128, 4, 4, False),
                                              (64, 2, 8, True), (64, 4, 2, False)])
def test_fused_norm_rope_append(gpu, d, bits, G, use_gain):
    rng = np.random.default_rng(100 + d + bits + G)
    B, H = 3, 2
    theta = 1e6 if d == 128 else 1e4
    gain = rng.uniform(0.5, 1.5, size=d) if use_gain else None
    say("norm+rope d=%d bits=%d G=%d gain=%s" % (d, bits, G, use_gain))
    p = Pair(gpu, B, H, G, d, bits, 4, 128, 8, 0.96, 0.92, cap=1100, symmetric=False, seed=3)
    for step, n in enumerate([[300, 0, 77], [1, 5, 16], [640, 2, 1], [3, 3, 3]]):
        k, v = _raw(rng, B, max(n), H, d)
        p.append_norm_rope(k, v, n, theta, gain=gain, eps=1e-6)
        p.check_cache()
        say(" step %d (n=%s)" % (step, n))
        _decode(p, _q(rng, B, H * G, d))
    _check_k_tilde(p)


def test_fused_norm_rope_eps_zero_and_large_positions(gpu):
    """eps = 0 (the paper's form of the RMS normalisation) and positions up
    to 8000 (angles far past 2 pi at the fastest rotary frequency)."""
    rng = np.random.default_rng(7)
    B, H, G, d = 1, 1, 4, 128
    p = Pair(gpu, B, H, G, d, 2, 4, 128, 8, 0.96, 0.92, cap=8200, seed=5)
    k, v = _raw(rng, B, 8000, H, d)
    p.append_norm_rope(k, v, [8000], 1e6, eps=0.0)
    p.check_cache()
    k, v = _raw(rng, B, 1, H, d)
    p.append_norm_rope(k, v, [1], 1e6, eps=0.0)
    p.check_cache()
    _decode(p, _q(rng, B, H * G, d))
    _check_k_tilde(p)
