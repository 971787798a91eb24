"""GPU parity: the HIP path through the C ABI against the oracle, at sizes
the oracle finishes in seconds (several pages, ragged tails)."""
import numpy as np
import pytest

from gpu_harness import Pair, rel_err, say, TOL
import oracle
from workloads import synth

pytestmark = pytest.mark.gpu


def _kv(rng, B, n, H, d, scale=1.0, outliers=()):
    k = rng.standard_normal((B, n, H, d)).astype(np.float32) * scale
    if len(outliers):
        k[..., list(outliers)] *= 8.0
    v = rng.standard_normal((B, n, H, d)).astype(np.float32)
    return oracle.f32_to_bf16(k), oracle.f32_to_bf16(v)


def _q(rng, B, nq, d):
    return oracle.f32_to_bf16(rng.standard_normal((B, nq, d)).astype(np.float32))


def test_tiny_config_prefill_then_decode_steps(gpu):
    """The tiny workload: one sequence, d = 64, 512-token context, then a
    run of single-token decode steps that crosses several flushes."""
    c = synth.CONFIGS["tiny"]
    w = synth.Workload(c)
    say("tiny: prefill 500")
    p = Pair(gpu, 1, 1, 4, 64, 2, c["s_sink"], c["s_keep"], c["s_flush"], c["kappa_k"],
             c["kappa_v"], cap=600)
    k = w.keys(0, 0, 512)[None]
    v = w.values(0, 0, 512)[None]
    p.append(k[:, :500], v[:, :500], [500])
    assert p.check_cache() > 0
    total, diff, bad = p.k_tilde_vs_ref()
    say("k~ vs fp64: %d of %d differ from the rounded exact product, %d outside the bound"
        % (diff, total, bad))
    assert bad == 0 and diff <= 1e-3 * total
    for step in range(12):
        say("tiny: step", step)
        p.append(k[:, 500 + step:501 + step], v[:, 500 + step:501 + step], [1])
        p.check_cache()
        _, em, er = p.decode_check(w.query(step))
        say("  rel err vs mirror %.2e, vs ref %.2e" % (em, er))


@pytest.mark.parametrize("d,bits,G,symmetric", [(128, 2, 4, True), (128, 4, 4, False),
                                                (64, 2, 8, False), (64, 4, 1, True),
                                                (128, 2, 2, False), (128, 2, 8, False),
                                                (128, 3, 4, False)])
def test_ragged_batches(gpu, d, bits, G, symmetric):
    rng = np.random.default_rng(d * 10 + bits + G)
    B, H = 3, 2
    say("ragged d=%d bits=%d G=%d sym=%s" % (d, bits, G, symmetric))
    p = Pair(gpu, B, H, G, d, bits, 4, 128, 8, 0.96, 0.92, cap=1200, symmetric=symmetric,
             seed=1)
    n1 = [0, 77, 333]
    k, v = _kv(rng, B, max(n1), H, d, outliers=(3, 17))
    p.append(k, v, n1)
    assert p.check_cache() > 0
    p.decode_check(_q(rng, B, H * G, d))
    n2 = [5, 1, 64]
    k, v = _kv(rng, B, max(n2), H, d, outliers=(3, 17))
    p.append(k, v, n2)
    p.check_cache()
    _, em, er = p.decode_check(_q(rng, B, H * G, d))
    say("  rel err vs mirror %.2e, vs ref %.2e" % (em, er))
    n3 = [700, 0, 400]
    k, v = _kv(rng, B, max(n3), H, d, outliers=(3, 17))
    p.append(k, v, n3)
    p.check_cache()
    p.decode_check(_q(rng, B, H * G, d))
    total, diff, bad = p.k_tilde_vs_ref()
    say("  k~ vs fp64: %d of %d differ from the rounded exact product, %d outside the bound"
        % (diff, total, bad))
    assert bad == 0 and diff <= 1e-3 * total


def test_odd_windows_and_partial_words(gpu):
    """s_flush = 5 and s_sink = 0: flushes end inside value-code words, so the
    writer must merge with what the page holds; no sink window at all."""
    rng = np.random.default_rng(7)
    B, H, G, d = 2, 1, 4, 128
    p = Pair(gpu, B, H, G, d, 2, 0, 7, 5, 0.9, 0.8, cap=400, win_slots=64)
    for step, n in enumerate([3, 1, 9, 1, 1, 40, 2, 1, 1, 1, 64, 7]):
        say("odd windows: step", step, "n", n)
        k, v = _kv(rng, B, n, H, d)
        p.append(k, v, [n, max(0, n - 1)])
        p.check_cache()
        p.decode_check(_q(rng, B, H * G, d))


def test_large_sink_and_split_flush(gpu):
    """A sink wider than a page and an append longer than the ring: the flush
    runs as its own launch before the new tokens reuse ring slots."""
    rng = np.random.default_rng(8)
    B, H, G, d = 2, 2, 4, 64
    p = Pair(gpu, B, H, G, d, 2, 70, 20, 4, 0.96, 0.92, cap=900, win_slots=128)
    for n in [50, 30, 1, 200, 3, 100]:
        say("large sink: append", n)
        k, v = _kv(rng, B, n, H, d)
        p.append(k, v, [n, n // 2])
        p.check_cache()
        p.decode_check(_q(rng, B, H * G, d))


def test_empty_and_short_sequences(gpu):
    rng = np.random.default_rng(9)
    B, H, G, d = 3, 1, 4, 64
    p = Pair(gpu, B, H, G, d, 2, 4, 16, 8, 0.96, 0.92, cap=200)
    say("empty: decode over nothing")
    out = p.decode(_q(rng, B, H * G, d))
    assert np.all(out == 0)
    k, v = _kv(rng, B, 3, H, d)
    p.append(k, v, [0, 3, 1])
    p.check_cache()
    out, _, _ = p.decode_check(_q(rng, B, H * G, d))
    assert np.all(out[0] == 0)


def test_needles_in_each_segment(gpu):
    """Plant one key aligned with the query, in the sink, the quantised
    middle (first, page boundary, last partial page) or the recent ring: the
    softmax mass lands on one segment and the output follows that token."""
    rng = np.random.default_rng(10)
    B, H, G, d = 1, 1, 4, 128
    S = 4 + 64 * 5 + 37 + 135  # several pages, a partial page, full windows
    for where in [1, 4, 67, 68, 4 + 64 * 5 + 30, S - 3]:
        say("needle at", where)
        p = Pair(gpu, B, H, G, d, 2, 4, 128, 8, 0.96, 0.92, cap=S + 8, symmetric=False)
        k, v = _kv(rng, B, S, H, d, scale=0.3)
        q = _q(rng, B, H * G, d)
        # k~ = T k should point along T^{-T} q, i.e. k = T^{-1} T^{-T} q
        T = oracle.bf16_to_f32(p.tk[0]).astype(np.float64)
        qf = oracle.bf16_to_f32(q[0, 0]).astype(np.float64)
        needle = np.linalg.solve(T, np.linalg.solve(T.T, qf))
        needle *= 6.0 / np.linalg.norm(T @ needle) * np.sqrt(d) / max(np.linalg.norm(qf), 1e-6)
        k[0, where, 0] = oracle.f32_to_bf16(needle.astype(np.float32))
        p.append(k, v, [S])
        p.check_cache()
        out, em, er = p.decode_check(q)
        say("  rel err %.2e %.2e" % (em, er))


def test_page_order_and_determinism(gpu):
    rng = np.random.default_rng(11)
    B, H, G, d = 2, 2, 4, 128
    outs = []
    for order in ("linear", "random"):
        p = Pair(gpu, B, H, G, d, 2, 4, 128, 8, 0.96, 0.92, cap=1500, page_order=order,
                 pool_factor=1.5, oracle_ref=False)
        r2 = np.random.default_rng(12)
        k, v = _kv(r2, B, 1400, H, d)
        say("page order", order)
        p.append(k, v, [1400, 999])
        q = _q(np.random.default_rng(13), B, H * G, d)
        a = p.decode(q)
        b = p.decode(q)
        assert np.array_equal(a, b), "decode is not deterministic"
        outs.append(a)
    assert np.array_equal(outs[0], outs[1]), "physical page order changed the result"


def test_dequant_bit_exact(gpu):
    import paper_2609_38121_amd as wk
    rng = np.random.default_rng(14)
    for d, bits in [(128, 2), (128, 4), (64, 2), (64, 4), (128, 3), (64, 3)]:
        B, H = 2, 2
        p = Pair(gpu, B, H, 4, d, bits, 4, 32, 8, 0.96, 0.92, cap=500, oracle_ref=False)
        k, v = _kv(rng, B, 450, H, d)
        p.append(k, v, [450, 200])
        m = p.mirror
        for b in range(B):
            qe = int(m.quant_end[b])
            say("dequant d=%d bits=%d b=%d [4,%d)" % (d, bits, b, qe))
            ko, vo = wk.wushkv_dequant(p.gpu, b, 4, qe - 4)
            ko, vo = ko.cpu().numpy(), vo.cpu().numpy()
            for h in range(H):
                kref = oracle.dequant(m.kc[b, h, 4:qe], m.kp[b, h, 4:qe, 0], m.kp[b, h, 4:qe, 1])
                vref = oracle.dequant(m.vc[b, h, 4:qe], m.vp[b, h, 4:qe, 0], m.vp[b, h, 4:qe, 1])
                assert np.array_equal(ko[h], kref)
                assert np.array_equal(vo[h], vref)
