"""GPU parity of the QuEST codec (Eq. (5), Sec. 4.3) through the C ABI: the
same append and decode entry points on a cache whose descriptor selects the
QuEST quantiser, against the oracle's QuEST cache (codes and fp16 parameters
bit for bit; decode within the row-normalised 2e-3 bar)."""
import numpy as np
import pytest

from gpu_harness import Pair, say
import oracle
from workloads import synth

pytestmark = pytest.mark.gpu


def _kv(rng, B, n, H, d, outliers=(3, 17)):
    k = rng.standard_normal((B, n, H, d)).astype(np.float32)
    k[..., list(outliers)] *= 8.0
    v = rng.standard_normal((B, n, H, d)).astype(np.float32)
    return oracle.f32_to_bf16(k), oracle.f32_to_bf16(v)


def _q(rng, B, nq, d):
    return oracle.f32_to_bf16(rng.standard_normal((B, nq, d)).astype(np.float32))


@pytest.mark.parametrize("d,bits,G", [(128, 2, 4), (128, 4, 1), (64, 2, 8), (64, 4, 2), (128, 3, 4),
                                     (64, 3, 2)])
def test_quest_ragged_prefill_and_steps(gpu, d, bits, G):
    rng = np.random.default_rng(100 + d + bits + G)
    B, H = 3, 2
    say("quest ragged d=%d bits=%d G=%d" % (d, bits, G))
    p = Pair(gpu, B, H, G, d, bits, 4, 64, 8, 0.96, 0.92, cap=1100, symmetric=(bits == 2),
             seed=2, codec="quest")
    n1 = [0, 150, 700]
    k, v = _kv(rng, B, max(n1), H, d)
    k[1, 70] = 0   # zero groups: Q(0) = 0
    v[2, 300] = 0
    p.append(k, v, n1)
    assert p.check_cache() > 0
    _, em, er = p.decode_check(_q(rng, B, H * G, d))
    say("  prefill: rel err vs mirror %.2e, vs ref %.2e" % (em, er))
    for step in range(10):  # single-token steps across flush boundaries
        k, v = _kv(rng, B, 1, H, d)
        p.append(k, v, [1, 1, 1])
        p.check_cache()
        p.decode_check(_q(rng, B, H * G, d))
    n3 = [200, 3, 90]
    k, v = _kv(rng, B, max(n3), H, d)
    p.append(k, v, n3)
    p.check_cache()
    _, em, er = p.decode_check(_q(rng, B, H * G, d))
    say("  after steps: rel err vs mirror %.2e, vs ref %.2e" % (em, er))
    # the zero groups (checked bit for bit against the mirror above) have
    # scale 0 and every code 2^(b-1), so they reconstruct to zero
    m = p.mirror
    assert np.all(m.kc[1, :, 70] == 2 ** (bits - 1)) and np.all(m.kp[1, :, 70, 0] == 0)
    assert np.all(m.vc[2, :, 300] == 2 ** (bits - 1)) and np.all(m.vp[2, :, 300, 0] == 0)


def test_quest_tiny_workload_decode_steps(gpu):
    c = synth.CONFIGS["tiny"]
    w = synth.Workload(c)
    say("quest tiny: prefill 500")
    p = Pair(gpu, 1, 1, 4, 64, 2, c["s_sink"], c["s_keep"], c["s_flush"], c["kappa_k"],
             c["kappa_v"], cap=600, codec="quest")
    k = w.keys(0, 0, 512)[None]
    v = w.values(0, 0, 512)[None]
    p.append(k[:, :500], v[:, :500], [500])
    assert p.check_cache() > 0
    for step in range(12):
        p.append(k[:, 500 + step:501 + step], v[:, 500 + step:501 + step], [1])
        p.check_cache()
        _, em, er = p.decode_check(w.query(step))
    say("  last step: rel err vs mirror %.2e, vs ref %.2e" % (em, er))


def test_quest_fused_norm_rope_prefill(gpu):
    """The Llama-shaped fused path (norm + RoPE + transform + QuEST) on two
    2048-token sequences of 8 heads."""
    rng = np.random.default_rng(101)
    B, H, G, d, S = 2, 8, 4, 128, 2048
    say("quest fused norm+rope prefill B=%d S=%d" % (B, S))
    p = Pair(gpu, B, H, G, d, 2, 4, 128, 8, 0.96, 0.92, cap=S + 64, codec="quest")
    k = oracle.f32_to_bf16((rng.standard_t(3.0, (B, S, H, d))).astype(np.float32))
    v = oracle.f32_to_bf16(rng.standard_normal((B, S, H, d)).astype(np.float32))
    p.append_norm_rope(k, v, [S, S - 333], theta=1e6)
    assert p.check_cache() > 0
    _, em, er = p.decode_check(_q(rng, B, H * G, d))
    say("  rel err vs mirror %.2e, vs ref %.2e" % (em, er))


def test_quest_dequant_bit_exact(gpu):
    import paper_2609_38121_amd as wk
    rng = np.random.default_rng(102)
    for d, bits in [(128, 2), (64, 4), (128, 3)]:
        B, H = 2, 2
        p = Pair(gpu, B, H, 4, d, bits, 4, 32, 8, 0.96, 0.92, cap=500, oracle_ref=False,
                 codec="quest")
        k, v = _kv(rng, B, 450, H, d)
        p.append(k, v, [450, 200])
        m = p.mirror
        for b in range(B):
            qe = int(m.quant_end[b])
            say("quest dequant d=%d bits=%d b=%d [4,%d)" % (d, bits, b, qe))
            ko, vo = wk.wushkv_dequant(p.gpu, b, 4, qe - 4)
            ko, vo = ko.cpu().numpy(), vo.cpu().numpy()
            for h in range(H):
                kref = oracle.dequant(m.kc[b, h, 4:qe], m.kp[b, h, 4:qe, 0], m.kp[b, h, 4:qe, 1])
                vref = oracle.dequant(m.vc[b, h, 4:qe], m.vp[b, h, 4:qe, 0], m.vp[b, h, 4:qe, 1])
                assert np.array_equal(ko[h], kref)
                assert np.array_equal(vo[h], vref)


@pytest.mark.parametrize("bits", [2, 3, 4])
def test_quest_library_default_alpha(gpu, bits):
    """A QuEST cache built without an explicit clip multiplier uses the
    library's alpha_b (wushkv_quest_alpha: the stationarity condition of the
    clipping lemma, App. B); it must be the oracle's Gaussian-optimal alpha_b
    (Sec. 4.3) within 1e-6, and the cache it builds must equal the oracle's
    QuEST cache at that same value bit for bit."""
    import paper_2609_38121_amd as wk
    rng = np.random.default_rng(110 + bits)
    B, H, G, d = 2, 2, 4, 128
    say("quest library-default alpha, bits=%d" % bits)
    p = Pair(gpu, B, H, G, d, bits, 4, 64, 8, 0.96, 0.92, cap=800, codec="quest",
             quest_alpha=None)
    lib_alpha = wk.wushkv_quest_alpha(bits)
    assert p.gpu.quest_alpha == float(np.float32(lib_alpha))
    assert abs(lib_alpha - oracle.quest_alpha(bits)) <= 1e-6 * lib_alpha
    k, v = _kv(rng, B, 600, H, d)
    p.append(k, v, [600, 257])
    assert p.check_cache() > 0
    _, em, er = p.decode_check(_q(rng, B, H * G, d))
    for _ in range(9):  # single-token steps across a flush
        k, v = _kv(rng, B, 1, H, d)
        p.append(k, v, [1, 1])
        p.check_cache()
        _, em, er = p.decode_check(_q(rng, B, H * G, d))
    say("  alpha %.7f: rel err vs mirror %.2e, vs ref %.2e" % (p.gpu.quest_alpha, em, er))
