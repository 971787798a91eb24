"""Pins of the oracle's cache management (Sec. 4.4, Alg. 2) and attention
(Eq. (2), Eq. (3)): hand-worked window examples, window invariants over
random schedules, flush-time independence, the transform-insertion identity,
and closed-form special cases of softmax attention."""
import os

import numpy as np
import pytest

import oracle
from workloads import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "windows_worked_examples.txt")


def _golden():
    rows = []
    for line in open(GOLDEN):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        head, chunks, expect = [p.strip() for p in line.split("|")]
        s_sink, s_keep, s_flush = (int(v) for v in head.split())
        cs = []
        for tok in chunks.split():
            if "*" in tok:
                a, n = tok.split("*")
                cs += [int(a)] * int(n)
            else:
                cs.append(int(tok))
        rows.append((s_sink, s_keep, s_flush, cs, [int(v) for v in expect.split()]))
    return rows


@pytest.mark.parametrize("row", _golden())
def test_window_worked_examples(row):
    s_sink, s_keep, s_flush, chunks, expect = row
    S, Q, got = 0, 0, []
    for n in chunks:
        S += n
        Q = oracle.next_quant_end(S, Q, s_sink, s_keep, s_flush)
        got.append(Q)
    if len(expect) == 1:
        got = got[-1:]
    assert got == expect


@pytest.mark.parametrize("s_sink,s_keep,s_flush", [(4, 128, 8), (16, 128, 16), (64, 256, 8),
                                                   (0, 5, 3), (7, 0, 1), (3, 10, 7)])
def test_window_invariants(s_sink, s_keep, s_flush):
    rng = np.random.default_rng(s_sink * 31 + s_keep * 7 + s_flush)
    for _ in range(50):
        S, Q = 0, 0
        for _ in range(60):
            n = int(rng.choice([0, 1, 1, 1, 2, 5, 17, 100]))
            S += n
            Qn = oracle.next_quant_end(S, Q, s_sink, s_keep, s_flush)
            assert Qn >= Q  # never un-quantises
            start = max(Q, s_sink)
            if Qn > start:
                assert (Qn - start) % s_flush == 0  # whole flushes only
            Q = Qn
            eff = max(Q, s_sink)
            assert Q <= max(S - s_keep, 0) or Q == 0 or Q <= s_sink
            if S >= s_sink + s_keep:
                # the recent window holds S_keep .. S_keep + S_flush - 1 entries
                assert s_keep <= S - eff < s_keep + s_flush
            else:
                assert eff <= max(S, s_sink)
            if Q > s_sink:
                assert (Q - s_sink) % s_flush == 0


def _state(cache):
    return (cache.kbits.copy(), cache.vbits.copy(), cache.kc.copy(), cache.vc.copy(),
            cache.kp.copy(), cache.vp.copy(), cache.seq_len.copy(), cache.quant_end.copy())


def _rand_bits(rng, shape, scale=1.0):
    return oracle.f32_to_bf16((rng.standard_normal(shape) * scale).astype(np.float32))


def test_flush_time_independence():
    rng = np.random.default_rng(3)
    B, H, d, n = 2, 2, 64, 300
    k = _rand_bits(rng, (B, n, H, d))
    v = _rand_bits(rng, (B, n, H, d))
    tk = _rand_bits(rng, (H, d, d), 0.2)
    kw = dict(batch=B, n_kv=H, d=d, bits=2, s_sink=4, s_keep=32, s_flush=8, kappa_k=0.96,
              kappa_v=0.92, capacity=n)
    one = oracle.OracleCache(**kw)
    one.append(k, v, np.array([n, n]), tk)
    many = oracle.OracleCache(**kw)
    t = 0
    for step in [1, 1, 3, 50, 1, 7, 100, 1, 1, 135]:
        many.append(k[:, t:t + step], v[:, t:t + step], np.array([step, step]), tk)
        t += step
    assert t == n
    for a, b in zip(_state(one), _state(many)):
        assert np.array_equal(a, b)


def test_eq3_identity_fp64():
    # attention on (T k, T^-T q) equals attention on (k, q) without rounding
    rng = np.random.default_rng(4)
    d, S = 64, 50
    for symmetric in (True, False):
        q1 = np.linalg.qr(rng.standard_normal((d, d)))[0]
        q2 = q1 if symmetric else np.linalg.qr(rng.standard_normal((d, d)))[0]
        T = (q1 * np.exp(rng.uniform(np.log(.5), np.log(2), d))) @ q2.T
        K = rng.standard_normal((S, d))
        V = rng.standard_normal((S, d))
        q = rng.standard_normal(d)
        ref = oracle.attend(q, K, V, 1 / 8)
        Kt = K @ T.T                      # rows T k
        qt = q @ np.linalg.inv(T)         # row form of T^{-T} q
        got = oracle.attend(qt, Kt, V, 1 / 8)
        assert np.max(np.abs(got - ref)) < 1e-12


def test_attention_special_cases():
    rng = np.random.default_rng(5)
    d = 32
    q = rng.standard_normal(d)
    # one token: output is its value
    K, V = rng.standard_normal((1, d)), rng.standard_normal((1, d))
    assert np.allclose(oracle.attend(q, K, V, 0.3), V[0], atol=0, rtol=0)
    # equal keys: output is the mean of the values
    K = np.repeat(rng.standard_normal((1, d)), 9, axis=0)
    V = rng.standard_normal((9, d))
    assert np.max(np.abs(oracle.attend(q, K, V, 0.3) - V.mean(axis=0))) < 1e-14
    # two tokens: logistic weight of the logit difference
    K, V = rng.standard_normal((2, d)), rng.standard_normal((2, d))
    l0, l1 = 0.3 * K[0] @ q, 0.3 * K[1] @ q
    w0 = 1.0 / (1.0 + np.exp(l1 - l0))
    assert np.max(np.abs(oracle.attend(q, K, V, 0.3) - (w0 * V[0] + (1 - w0) * V[1]))) < 1e-14
    # a planted key with a huge logit takes all the mass
    K = rng.standard_normal((40, d))
    K[17] = q * 50
    V = rng.standard_normal((40, d))
    assert np.max(np.abs(oracle.attend(q, K, V, 1.0) - V[17])) < 1e-12
    # permutation invariance
    perm = rng.permutation(40)
    K = rng.standard_normal((40, d))
    assert np.max(np.abs(oracle.attend(q, K, V, 0.2) - oracle.attend(q, K[perm], V[perm], 0.2))) < 1e-13
    # empty cache gives zeros
    assert np.all(oracle.attend(q, np.zeros((0, d)), np.zeros((0, d)), 0.2) == 0)


def test_decode_head_on_windows_only_equals_plain_attention():
    # S <= S_sink + S_keep: nothing is quantised, so decode over the cache is
    # attention over bf16(T k) with the compensated query (Eq. (3)) -- equal
    # to plain attention up to the bf16 rounding of T k.
    rng = np.random.default_rng(6)
    B, H, G, d, n = 1, 1, 4, 64, 30
    k = _rand_bits(rng, (B, n, H, d))
    v = _rand_bits(rng, (B, n, H, d))
    Tf = np.linalg.qr(rng.standard_normal((d, d)))[0] * 1.3
    tk = oracle.f32_to_bf16(Tf.astype(np.float32))[None]
    Tb = oracle.bf16_to_f32(tk[0]).astype(np.float64)
    tinv = np.linalg.inv(Tb).astype(np.float32)[None]
    cache = oracle.OracleCache(B, H, d, 2, 4, 32, 8, 0.96, 0.92, n)
    cache.append(k, v, np.array([n]), tk)
    assert cache.quant_end[0] == 0
    q = _rand_bits(rng, (B, G, d))
    out = cache.decode(q, tinv, 1 / 8)
    K = oracle.bf16_to_f32(k[0, :, 0]).astype(np.float64)
    V = oracle.bf16_to_f32(v[0, :, 0]).astype(np.float64)
    for g in range(G):
        ref = oracle.attend(oracle.bf16_to_f32(q[0, g]).astype(np.float64), K, V, 1 / 8)
        assert np.max(np.abs(out[0, g] - ref)) < 2e-2 * np.max(np.abs(ref))


def test_decode_head_brute_force_tiny():
    # decode over a quantised cache equals explicit softmax over the
    # reconstructed rows, built here element by element
    rng = np.random.default_rng(7)
    B, H, G, d, n = 1, 1, 2, 64, 60
    k = _rand_bits(rng, (B, n, H, d))
    v = _rand_bits(rng, (B, n, H, d))
    tk = oracle.f32_to_bf16(np.eye(d, dtype=np.float32))[None]
    tinv = np.eye(d, dtype=np.float32)[None]
    cache = oracle.OracleCache(B, H, d, 2, 4, 16, 8, 0.96, 0.92, n)
    cache.append(k, v, np.array([n]), tk)
    S, Q = int(cache.seq_len[0]), int(cache.quant_end[0])
    assert Q > 4
    q = _rand_bits(rng, (B, G, d))
    out = cache.decode(q, tinv, 0.125)
    for g in range(G):
        qq = [float(oracle.bf16_to_f32(q[0, g, i])) for i in range(d)]
        logits, rows = [], []
        for p in range(S):
            if 4 <= p < Q:
                s = float(oracle.f16_to_f32(cache.kp[0, 0, p, 0]))
                z = float(oracle.f16_to_f32(cache.kp[0, 0, p, 1]))
                kr = [s * int(cache.kc[0, 0, p, i]) + z for i in range(d)]
                s = float(oracle.f16_to_f32(cache.vp[0, 0, p, 0]))
                z = float(oracle.f16_to_f32(cache.vp[0, 0, p, 1]))
                vr = [s * int(cache.vc[0, 0, p, i]) + z for i in range(d)]
            else:
                kr = [float(oracle.bf16_to_f32(cache.kbits[0, 0, p, i])) for i in range(d)]
                vr = [float(oracle.bf16_to_f32(cache.vbits[0, 0, p, i])) for i in range(d)]
            logits.append(0.125 * sum(a * b for a, b in zip(qq, kr)))
            rows.append(vr)
        m = max(logits)
        w = [np.exp(x - m) for x in logits]
        ref = [sum(w[p] * rows[p][i] for p in range(S)) / sum(w) for i in range(d)]
        assert np.max(np.abs(out[0, g] - np.array(ref))) < 1e-12


def test_chunk_attention_brute_force_causal():
    """Chunk attention (Alg. 2 step 5 with S' > 1): token t of the chunk sees
    positions up to its own and no later one.  Checked against an explicit
    causal softmax over the reconstructed rows, built element by element, and
    the chunk's last token against decode."""
    rng = np.random.default_rng(8)
    B, H, G, d, n0, T = 2, 1, 2, 64, 70, 5
    tk = oracle.f32_to_bf16(np.eye(d, dtype=np.float32))[None]
    tinv = np.eye(d, dtype=np.float32)[None]
    cache = oracle.OracleCache(B, H, d, 2, 4, 16, 8, 0.96, 0.92, n0 + T)
    k = _rand_bits(rng, (B, n0, H, d))
    v = _rand_bits(rng, (B, n0, H, d))
    cache.append(k, v, np.array([n0, n0 - 9]), tk)
    k = _rand_bits(rng, (B, T, H, d))
    v = _rand_bits(rng, (B, T, H, d))
    n_tok = np.array([T, 3])
    cache.append(k, v, n_tok, tk)
    q = _rand_bits(rng, (B, T, G * H, d))
    out = oracle.chunk_attention(cache, q, n_tok, tinv, 0.125)
    for b in range(B):
        S, Q = int(cache.seq_len[b]), int(cache.quant_end[b])
        assert Q > 4
        n = int(n_tok[b])
        assert np.all(np.isnan(out[b, n:]))
        for t in range(n):
            last = S - n + t  # the position of this token
            for g in range(G):
                qq = [float(oracle.bf16_to_f32(q[b, t, g, i])) for i in range(d)]
                logits, rows = [], []
                for p in range(last + 1):
                    if 4 <= p < Q:
                        s = float(oracle.f16_to_f32(cache.kp[b, 0, p, 0]))
                        z = float(oracle.f16_to_f32(cache.kp[b, 0, p, 1]))
                        kr = [s * int(cache.kc[b, 0, p, i]) + z for i in range(d)]
                        s = float(oracle.f16_to_f32(cache.vp[b, 0, p, 0]))
                        z = float(oracle.f16_to_f32(cache.vp[b, 0, p, 1]))
                        vr = [s * int(cache.vc[b, 0, p, i]) + z for i in range(d)]
                    else:
                        kr = [float(oracle.bf16_to_f32(cache.kbits[b, 0, p, i])) for i in range(d)]
                        vr = [float(oracle.bf16_to_f32(cache.vbits[b, 0, p, i])) for i in range(d)]
                    logits.append(0.125 * sum(a * c for a, c in zip(qq, kr)))
                    rows.append(vr)
                m = max(logits)
                w = [np.exp(x - m) for x in logits]
                ref = [sum(w[p] * rows[p][i] for p in range(last + 1)) / sum(w) for i in range(d)]
                assert np.max(np.abs(out[b, t, g] - np.array(ref))) < 1e-12
    # the last token of each chunk attends to everything: that is decode
    q_last = np.stack([q[b, int(n_tok[b]) - 1] for b in range(B)])
    dec = cache.decode(q_last, tinv, 0.125)
    for b in range(B):
        assert np.array_equal(dec[b], out[b, int(n_tok[b]) - 1])


def _brute_decode(cache, b, h, q_row, S, Q, scale):
    """Softmax attention of one bf16 query over positions [0, S) of (b, h):
    positions in [s_sink, Q) through their codes, the others at bf16, every
    row rebuilt here from the stored codes and parameters."""
    d = cache.d
    qq = oracle.bf16_to_f32(q_row).astype(np.float64)
    logits, rows = [], []
    for p in range(S):
        if cache.s_sink <= p < Q:
            s, z = (float(oracle.f16_to_f32(x)) for x in cache.kp[b, h, p])
            kr = s * cache.kc[b, h, p].astype(np.float64) + z
            s, z = (float(oracle.f16_to_f32(x)) for x in cache.vp[b, h, p])
            vr = s * cache.vc[b, h, p].astype(np.float64) + z
        else:
            kr = oracle.bf16_to_f32(cache.kbits[b, h, p]).astype(np.float64)
            vr = oracle.bf16_to_f32(cache.vbits[b, h, p]).astype(np.float64)
        logits.append(scale * float(qq @ kr))
        rows.append(vr)
    w = np.exp(np.array(logits) - max(logits))
    return (w[:, None] * np.array(rows)).sum(axis=0) / w.sum()


def test_decode_step_order_of_alg2():
    # a run of single-token steps crossing flushes: each step's attention
    # sees the positions its own flush quantises at bf16 (Alg. 2 quantises
    # after step 5), and equals append + decode exactly on steps that flush
    # nothing; the cache ends as after the plain appends
    rng = np.random.default_rng(21)
    B, H, G, d, n0, steps = 2, 1, 2, 64, 40, 14
    k = _rand_bits(rng, (B, n0 + steps, H, d))
    v = _rand_bits(rng, (B, n0 + steps, H, d))
    tk = oracle.f32_to_bf16(np.eye(d, dtype=np.float32))[None]
    tinv = np.eye(d, dtype=np.float32)[None]
    kw = dict(batch=B, n_kv=H, d=d, bits=2, s_sink=4, s_keep=16, s_flush=8, kappa_k=0.96,
              kappa_v=0.92, capacity=n0 + steps)
    fused, plain = oracle.OracleCache(**kw), oracle.OracleCache(**kw)
    for c in (fused, plain):
        c.append(k[:, :n0], v[:, :n0], np.array([n0, n0 - 3]), tk)
    flushes = 0
    for t in range(steps):
        n_new = np.array([1, t % 3 != 0])  # sequence 1 skips some steps
        q = _rand_bits(rng, (B, H * G, d))
        q_old, s_old = fused.quant_end.copy(), fused.seq_len.copy()
        pos = s_old.copy()
        kn = np.stack([k[b, pos[b], :] for b in range(B)])
        vn = np.stack([v[b, pos[b], :] for b in range(B)])
        got = oracle.decode_step(fused, kn, vn, n_new, tk, q, tinv, 0.125)
        plain.append(kn[:, None], vn[:, None], n_new, tk)
        ref = plain.decode(q, tinv, 0.125)
        for a, b in zip(_state(fused), _state(plain)):
            assert np.array_equal(a, b)
        for b in range(B):
            S = int(s_old[b] + n_new[b])
            for g in range(G):
                want = _brute_decode(fused, b, 0, q[b, g], S, int(q_old[b]), 0.125)
                assert np.max(np.abs(got[b, g] - want)) < 1e-12
            if fused.quant_end[b] == q_old[b]:
                assert np.array_equal(got[b], ref[b])
            else:
                flushes += 1
                assert not np.array_equal(got[b], ref[b])
    assert flushes >= 2


def test_parallel_pairs_equal_the_serial_oracle():
    """The benchmark's OpenMP driver (HeadSet: independent (sequence, head)
    pairs spread over threads) computes exactly what OracleCache computes
    pair by pair: same codes, parameters, counters and decode outputs, bit
    for bit, at any thread count."""
    rng = np.random.default_rng(77)
    d, G, bits = 64, 4, 2
    lens = [300, 0, 41, 130, 257]
    tk, tinv = synth.make_transform(len(lens), d, 5, False)
    hs = {}
    for threads in (1, 3):
        h = oracle.HeadSet([n + 8 for n in lens], d, bits, 4, 32, 8, 0.96, 0.92)
        ks = [oracle.f32_to_bf16(rng.standard_normal((n, d)).astype(np.float32)) for n in lens]
        vs = [oracle.f32_to_bf16(rng.standard_normal((n, d)).astype(np.float32)) for n in lens]
        if threads == 1:
            inputs = (ks, vs)
        ks, vs = inputs
        used = h.append(ks, vs, [tk[i] for i in range(len(lens))], threads=threads)
        assert used == threads
        qs = [oracle.f32_to_bf16(np.random.default_rng(i).standard_normal((G, d)).astype(np.float32))
              for i in range(len(lens))]
        out, used = h.decode(qs, [tinv[i] for i in range(len(lens))], 0.125, threads=threads)
        assert used == threads
        hs[threads] = (h, out)
        for i, n in enumerate(lens):
            oc = oracle.OracleCache(1, 1, d, bits, 4, 32, 8, 0.96, 0.92, n + 8)
            oc.append(ks[i][None, :, None], vs[i][None, :, None], [n], tk[i:i + 1])
            assert int(oc.seq_len[0]) == h.seq_len[i] and int(oc.quant_end[0]) == h.quant_end[i]
            assert np.array_equal(oc.kc[0, 0], h.kc[i]) and np.array_equal(oc.vc[0, 0], h.vc[i])
            assert np.array_equal(oc.kp[0, 0], h.kp[i]) and np.array_equal(oc.vp[0, 0], h.vp[i])
            ref = oc.decode(qs[i][None], tinv[i:i + 1], 0.125)[0]
            assert np.array_equal(ref, out[i]) or (n == 0 and np.all(out[i] == 0))
    assert np.array_equal(hs[1][1], hs[3][1])
