"""GPU parity of the append's two ways of advancing S and S_quant (Alg. 2
steps 4 and 7-11): a launch of at most 64 workgroups per sequence counts its
arrivals in the commit array and its last workgroup writes the counters; a
larger one counts none and a one-workgroup launch after it writes them.
Appends on both sides of that boundary, one after another on the same cache
and with ragged and zero counts, keep the cache bit-exact with the mirror
and the counters equal to the oracle's, take the path their size calls for,
and leave the commit array zero."""
import numpy as np
import pytest

import oracle
import paper_2609_38121_amd as wk
from gpu_harness import Pair, say

pytestmark = pytest.mark.gpu


def _kv(rng, B, n, H, d):
    k = rng.standard_normal((B, n, H, d)).astype(np.float32)
    k[..., [5, 40]] *= 6.0
    v = rng.standard_normal((B, n, H, d)).astype(np.float32)
    return oracle.f32_to_bf16(k), oracle.f32_to_bf16(v)


def _append_launches(p, k, v, counts):
    wk.wushkv_timing_enable(64)
    try:
        p.append(k, v, counts)
        names = [nm for nm, _ in wk.wushkv_timing_launches()]
    finally:
        wk.wushkv_timing_enable(0)
    return names


@pytest.mark.parametrize("d,bits,G", [(128, 2, 4), (64, 4, 2)])
def test_counter_commit_paths(gpu, d, bits, G):
    rng = np.random.default_rng(11 + d + bits)
    B, H = 3, 8
    p = Pair(gpu, B, H, G, d, bits, 4, 128, 8, 0.96, 0.92, cap=2400, seed=3)
    # (counts, whether the counters take a launch of their own): 8 kv heads
    # and a grid of 8 tiles make 64 workgroups per sequence, 16 tiles 128
    plan = [([20, 0, 33], False), ([700, 650, 0], True), ([40, 17, 90], False),
            ([0, 900, 310], True), ([25, 25, 25], False)]
    for counts, own_launch in plan:
        counts = np.array(counts, np.int32)
        k, v = _kv(rng, B, int(counts.max()), H, d)
        names = _append_launches(p, k, v, counts)
        say("append %s: launches %s" % (counts.tolist(), names))
        assert ("append_commit" in names) == own_launch, names
        n_codes = p.check_cache()
        assert np.array_equal(p.gpu.seq_len.cpu().numpy(), p.ref.seq_len)
        assert np.array_equal(p.gpu.quant_end.cpu().numpy(), p.ref.quant_end)
        assert np.all(p.gpu.commit.cpu().numpy() == 0)
        say("  S %s, S_quant %s, %d codes bit-exact" % (p.ref.seq_len.tolist(), p.ref.quant_end.tolist(), n_codes))
