"""GPU parity of the fused decode step (wushkv_decode_step): Alg. 2 for one
new token per sequence in the algorithm's own order (append, attention with
the positions due for quantisation still at bf16, then the flush), against
the oracle's decode_step; against the separate append + decode calls, with
which it must agree bit for bit on every step that quantises nothing; and at
the full Llama-shaped size on sampled heads."""
import numpy as np
import pytest
import torch

import oracle
import pagelayout
import paper_2609_38121_amd as wk
from gpu_harness import Pair, TOL, rel_err, say, to_dev_bf16, to_np_bits
from workloads import synth

pytestmark = pytest.mark.gpu


def _kv(rng, B, n, H, d, outliers=()):
    k = rng.standard_normal((B, n, H, d)).astype(np.float32)
    if len(outliers):
        k[..., list(outliers)] *= 8.0
    v = rng.standard_normal((B, n, H, d)).astype(np.float32)
    return oracle.f32_to_bf16(k), oracle.f32_to_bf16(v)


def _q(rng, B, nq, d):
    return oracle.f32_to_bf16(rng.standard_normal((B, nq, d)).astype(np.float32))


@pytest.mark.parametrize("d,bits,G,codec", [(128, 2, 4, "pclip"), (128, 4, 8, "pclip"),
                                            (64, 2, 1, "pclip"), (64, 4, 2, "quest"),
                                            (128, 2, 4, "quest"), (128, 3, 4, "quest"),
                                            (64, 3, 8, "pclip")])
def test_step_across_flushes(gpu, d, bits, G, codec):
    """Single-token steps from an empty sequence (sink slots), a short one
    and a long one, with some sequences skipping steps, across several
    flushes: the cache stays bit-exact with the mirror and every output
    matches the oracle's step."""
    rng = np.random.default_rng(300 + d + bits + G)
    B, H = 3, 2
    say("step d=%d bits=%d G=%d codec=%s" % (d, bits, G, codec))
    p = Pair(gpu, B, H, G, d, bits, 4, 16, 8, 0.96, 0.92, cap=600, seed=2, codec=codec)
    n0 = [0, 21, 333]
    k, v = _kv(rng, B, max(n0), H, d, outliers=(5,))
    p.append(k, v, n0)
    flushes = 0
    for t in range(30):
        n_new = [1, 1 if t % 4 else 0, 1]
        k1, v1 = _kv(rng, B, 1, H, d, outliers=(5,))
        q_old = p.mirror.quant_end.copy()
        _, em, er = p.step(k1[:, 0], v1[:, 0], n_new, _q(rng, B, H * G, d))
        p.check_cache()
        flushes += int(np.count_nonzero(p.mirror.quant_end != q_old))
        if t % 10 == 9:
            say("  step %d: rel err vs mirror %.2e, vs ref %.2e" % (t, em, er))
    assert flushes >= 6
    total, diff, bad = p.k_tilde_vs_ref()
    say("  k~ vs fp64: %d of %d differ from the rounded exact product, %d outside the bound"
        % (diff, total, bad))
    assert bad == 0 and diff <= 1e-3 * total


def test_step_equals_append_then_decode(gpu):
    """The same inputs through the fused step and through append + decode:
    the caches are identical after every step and the outputs identical on
    every step that quantises nothing."""
    rng = np.random.default_rng(31)
    B, H, G, d = 2, 2, 4, 128
    a = Pair(gpu, B, H, G, d, 2, 4, 64, 8, 0.96, 0.92, cap=1200, seed=3, oracle_ref=False)
    b = Pair(gpu, B, H, G, d, 2, 4, 64, 8, 0.96, 0.92, cap=1200, seed=3, oracle_ref=False)
    k, v = _kv(rng, B, 700, H, d)
    for p in (a, b):
        p.append(k, v, [700, 650])
    same = differ = 0
    for t in range(20):
        k1, v1 = _kv(rng, B, 1, H, d)
        q = _q(rng, B, H * G, d)
        q_old = b.mirror.quant_end.copy()
        got, _, _ = a.step(k1[:, 0], v1[:, 0], [1, 1], q, max_seq_len=1200)
        b.append(k1, v1, [1, 1])
        want = b.decode(q, max_seq_len=1200)
        for x, y in zip(a.host_state(), b.host_state()):
            assert np.array_equal(x, y), "caches differ after step %d" % t
        for s in range(B):
            if b.mirror.quant_end[s] == q_old[s]:
                assert np.array_equal(got[s], want[s]), "step %d sequence %d" % (t, s)
                same += 1
            else:
                differ += 1
    say("  %d sequence-steps equal, %d flushing" % (same, differ))
    assert same >= 30 and differ >= 4


def _mirror_pair(state, b, h, cfg, cap):
    """An oracle cache for (sequence b, kv head h) rebuilt from a host copy of
    the GPU cache: codes and params of the quantised positions from the
    pages, bf16 patterns of the sink and ring positions from the windows."""
    pages, table, win_k, win_v, seq_len, quant_end = state
    d, bits, s_sink = cfg["d"], cfg["bits"], cfg["s_sink"]
    m = oracle.OracleCache(1, 1, d, bits, s_sink, cfg["s_keep"], cfg["s_flush"], cfg["kappa_k"],
                           cfg["kappa_v"], cap)
    S, Q = int(seq_len[b]), int(quant_end[b])
    qe = max(Q, s_sink)
    if qe > s_sink:
        kc, vc, kp, vp = pagelayout.gather_sequence(pages, table, b, h, cfg["n_kv"], d, bits,
                                                    s_sink, qe)
        m.kc[0, 0, s_sink:qe], m.vc[0, 0, s_sink:qe] = kc, vc
        m.kp[0, 0, s_sink:qe], m.vp[0, 0, s_sink:qe] = kp, vp
    ring = win_k.shape[2] - s_sink
    for p in list(range(min(S, s_sink))) + list(range(qe, S)):
        slot = p if p < s_sink else s_sink + (p - s_sink) % ring
        m.kbits[0, 0, p] = win_k[b, h, slot]
        m.vbits[0, 0, p] = win_v[b, h, :, slot]
    m.seq_len[0], m.quant_end[0] = S, Q
    return m


@pytest.mark.timeout(900)
def test_step_llama_shaped(gpu):
    """The Llama-shaped decode workload (8 sequences, 8 kv heads, 32 query
    heads, 8192-token context, 2-bit) stepped 12 times by the fused call and
    by append + decode: identical caches throughout, identical outputs on the
    steps that flush nothing, and on the flushing steps sampled heads match
    the oracle's step on a mirror rebuilt from the GPU's cache."""
    cfg = dict(synth.CONFIGS["llama8b"])
    w = synth.Workload(cfg, seed=0)
    B, H, NQ, D = cfg["batch"], cfg["n_kv"], cfg["n_q"], cfg["d"]
    G, ctx, cap = NQ // H, cfg["ctx"], cfg["ctx"] + 64
    say("llama step: generating %d x %d tokens" % (B, ctx))
    k = np.stack([w.keys(b, 0, ctx) for b in range(B)])
    v = np.stack([w.values(b, 0, ctx) for b in range(B)])
    tk, tinv = w.transform()
    tk_d, tinv_d = to_dev_bf16(tk, gpu), torch.from_numpy(tinv).to(gpu)
    fused = wk.WushKVCache(B, H, D, cfg["bits"], cfg["s_sink"], cfg["s_keep"], cfg["s_flush"],
                           cfg["kappa_k"], cfg["kappa_v"], max_seq_len=cap, device=gpu)
    wk.wushkv_append(fused, to_dev_bf16(k, gpu), to_dev_bf16(v, gpu),
                     torch.full((B,), ctx, dtype=torch.int32, device=gpu), tk_d)
    torch.cuda.synchronize()
    del k, v
    plain = fused.clone()
    ones = torch.ones(B, dtype=torch.int32, device=gpu)
    sm = 1.0 / np.sqrt(D)
    pairs = [(0, 0), (3, 5), (7, 7)]
    eye = oracle.f32_to_bf16(np.eye(D, dtype=np.float32))[None]
    flushing = 0
    for t in range(12):
        say("llama step", t)
        k1 = np.stack([w.keys(b, ctx + t, 1)[0] for b in range(B)])
        v1 = np.stack([w.values(b, ctx + t, 1)[0] for b in range(B)])
        q = w.query(t)
        before = (fused.pages.cpu().numpy(), fused.page_table.cpu().numpy(), to_np_bits(fused.win_k),
                  to_np_bits(fused.win_v), fused.seq_len.cpu().numpy(), fused.quant_end.cpu().numpy())
        got = wk.wushkv_decode_step(fused, to_dev_bf16(k1, gpu), to_dev_bf16(v1, gpu), ones, tk_d,
                                    to_dev_bf16(q, gpu), tinv_d, sm_scale=sm, max_seq_len=cap)
        wk.wushkv_append(plain, to_dev_bf16(k1[:, None], gpu), to_dev_bf16(v1[:, None], gpu),
                         ones, tk_d)
        want = wk.wushkv_decode_attention(plain, to_dev_bf16(q, gpu), tinv_d, sm_scale=sm,
                                          max_seq_len=cap)
        torch.cuda.synchronize()
        for name in ("pages", "win_k", "win_v", "seq_len", "quant_end"):
            assert torch.equal(getattr(fused, name), getattr(plain, name)), (name, t)
        got, want = got.cpu().numpy(), want.cpu().numpy()
        qe = fused.quant_end.cpu().numpy()
        win_k = to_np_bits(fused.win_k)
        for b in range(B):
            if qe[b] == before[5][b]:
                assert np.array_equal(got[b], want[b]), (t, b)
                continue
            flushing += 1
            for (pb, h) in pairs:
                if pb != b:
                    continue
                m = _mirror_pair(before, b, h, cfg, cap)
                p = int(before[4][b])
                ring = fused.win_slots - cfg["s_sink"]
                kt = win_k[b, h, cfg["s_sink"] + (p - cfg["s_sink"]) % ring][None, None]
                ref = oracle.decode_step(m, kt, v1[b, h][None, None], np.array([1]), eye,
                                         q[b, h * G:(h + 1) * G][None], tinv[h][None], sm)
                e = rel_err(got[b, h * G:(h + 1) * G], ref[0])
                say("  step %d (b=%d, h=%d) flushing: rel err vs oracle %.2e" % (t, b, h, e))
                assert e <= TOL
    assert flushing >= 8


@pytest.mark.parametrize("s_flush,codec", [(5, "pclip"), (3, "quest"), (8, "pclip")])
def test_short_flushes_end_inside_value_words(gpu, s_flush, codec):
    """Flushes of s_flush = 3 or 5 positions end inside value-code words (8
    tokens each), so the short-flush quantiser (16 lanes per group) must
    merge its codes with what the page holds; single-token appends and fused
    steps alternate, over ragged sequences, and the caches stay bit-exact."""
    rng = np.random.default_rng(400 + s_flush)
    B, H, G, d = 3, 2, 4, 128
    say("short flushes s_flush=%d codec=%s" % (s_flush, codec))
    p = Pair(gpu, B, H, G, d, 2, 4, 16, s_flush, 0.96, 0.92, cap=400, seed=4, codec=codec)
    k, v = _kv(rng, B, 60, H, d)
    p.append(k, v, [60, 23, 0])
    flushes = 0
    for t in range(40):
        n_new = [1, 1, 1 if t % 3 else 0]
        k1, v1 = _kv(rng, B, 1, H, d)
        q_old = p.mirror.quant_end.copy()
        if t % 2:
            p.step(k1[:, 0], v1[:, 0], n_new, _q(rng, B, H * G, d))
        else:
            p.append(k1, v1, n_new)
            p.decode_check(_q(rng, B, H * G, d))
        p.check_cache()
        flushes += int(np.count_nonzero(p.mirror.quant_end != q_old))
    say("  %d flushes" % flushes)
    assert flushes >= 10
