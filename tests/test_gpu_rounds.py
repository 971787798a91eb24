"""GPU parity of the round-based decode: batches with so many (sequence, kv
head) pairs that the decode grid cannot be resident at once, so q~ comes from
decode_qt_kernel and each row has one window workgroup walking all its
window units.  Every head is checked against the oracle on the
GPU's own cache (mirror) and from the raw inputs (reference, the GPU's k~
substituted at rounding-tie positions), with empty, sink-only, one-page,
page-aligned and ragged sequences, and with two split plans (another
max_seq_len changes the page runs, odd or even in length, and only the fp32
summation order)."""
import numpy as np
import pytest

import oracle
import paper_2609_38121_amd as wk
from gpu_harness import Pair, TOL, rel_err, say

pytestmark = pytest.mark.gpu

SPLIT_TOL = 1e-5


def _kv(rng, B, n, H, d):
    k = rng.standard_normal((B, n, H, d)).astype(np.float32)
    k[..., [3, 17]] *= 8.0
    v = rng.standard_normal((B, n, H, d)).astype(np.float32)
    return oracle.f32_to_bf16(k), oracle.f32_to_bf16(v)


def _launched(p, q):
    wk.wushkv_timing_enable(64)
    try:
        p.decode(q)
        names = [nm for nm, _ in wk.wushkv_timing_launches()]
    finally:
        wk.wushkv_timing_enable(0)
    return names


@pytest.mark.parametrize("d,bits,G", [(128, 2, 4), (128, 4, 4), (64, 2, 8)])
def test_round_based_decode_every_head(gpu, d, bits, G):
    rng = np.random.default_rng(31 + d + bits + G)
    B, H = 48, 8
    lens = rng.integers(0, 2200, B)
    lens[:6] = [0, 1, 4, 132, 196, 64 * 20 + 4]
    say("rounds: batch %d, %d kv heads, G %d, d %d, %d-bit, lengths %d..%d"
        % (B, H, G, d, bits, lens.min(), lens.max()))
    p = Pair(gpu, B, H, G, d, bits, 4, 128, 8, 0.96, 0.92, cap=int(lens.max()) + 64, seed=7)
    k, v = _kv(rng, B, int(lens.max()), H, d)
    p.append(k, v, lens)
    q = oracle.f32_to_bf16(rng.standard_normal((B, H * G, d)).astype(np.float32))
    names = _launched(p, q)
    assert "decode_qt_kernel" in names, names  # the grid runs in rounds
    out = p.decode(q)
    assert np.all(np.isfinite(out))
    assert np.all(out[lens == 0] == 0)
    em = rel_err(out, p.mirror.decode(q, p.tinv, p.sm_scale))
    ref, n_sub = p.reference_for(lambda cache: cache.decode(q, p.tinv, p.sm_scale))
    er = rel_err(out, ref)
    say("  rel err vs mirror %.2e, vs reference %.2e (%d tie positions substituted)" % (em, er, n_sub))
    assert em <= TOL, "decode vs oracle on the GPU's cache: %.3e" % em
    assert er <= TOL, "decode vs oracle from raw inputs: %.3e" % er
    for extra in (64, 640):
        other = p.decode(q, max_seq_len=int(lens.max()) + extra)
        es = rel_err(other, out)
        say("  max_seq_len + %d: rel diff %.2e" % (extra, es))
        assert es <= SPLIT_TOL
