"""A token's stored key k~ = T_K k (Alg. 2 step 3), and so its codes, does not
depend on the path that formed it.  The prefill tiles (more than 16 new
tokens per call), short appends (at most 16) and the fused decode step all
form k~ with the same matrix-instruction operands (the shared key tile), and
the fused normalisation + RoPE with the same row code, so the same tokens
appended in one call, in short calls or by decode steps leave byte-identical
caches and identical k~ outputs."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_38121_amd as wk
from gpu_harness import say, to_dev_bf16, to_np_bits
from workloads import synth

pytestmark = pytest.mark.gpu

S_SINK, S_KEEP, S_FLUSH = 4, 32, 8


def _cache(gpu, B, H, d, bits, cap):
    return wk.WushKVCache(B, H, d, bits, S_SINK, S_KEEP, S_FLUSH, 0.96, 0.92, max_seq_len=cap,
                          device=gpu)


def _append(c, k, v, n, tk, table=None):
    """One append call; returns its k~ output (bf16 patterns)."""
    kd, vd = to_dev_bf16(k, c.device), to_dev_bf16(v, c.device)
    nd = torch.from_numpy(np.asarray(n, np.int32)).to(c.device)
    kt = torch.full_like(kd, float("nan"))
    if table is None:
        wk.wushkv_append(c, kd, vd, nd, tk, k_tilde_out=kt)
    else:
        wk.wushkv_append_norm_rope(c, kd, vd, nd, tk, table, norm_eps=1e-6, k_tilde_out=kt)
    torch.cuda.synchronize()
    return to_np_bits(kt)


def _state(c):
    """Counters, the page pool and the live window slots of every sequence."""
    torch.cuda.synchronize()
    seq, qe = c.seq_len.cpu().numpy(), c.quant_end.cpu().numpy()
    win_k, win_v = to_np_bits(c.win_k), to_np_bits(c.win_v)
    ring = c.win_slots - S_SINK
    live_k, live_v = [], []
    for b in range(c.batch):
        hi = max(int(qe[b]), S_SINK)
        for p in list(range(min(int(seq[b]), S_SINK))) + list(range(hi, int(seq[b]))):
            slot = p if p < S_SINK else S_SINK + (p - S_SINK) % ring
            live_k.append(win_k[b, :, slot])
            live_v.append(win_v[b, :, :, slot])
    return seq, qe, c.pages.cpu().numpy(), np.array(live_k), np.array(live_v)


def _same_state(a, b, what):
    for x, y, name in zip(_state(a), _state(b), ("seq_len", "quant_end", "pages", "win_k", "win_v")):
        assert np.array_equal(x, y), "%s: %s differs" % (what, name)


@pytest.mark.parametrize("d,bits,fused_norm", [(128, 2, False), (128, 4, True), (64, 2, True),
                                               (64, 4, False)])
def test_prefill_short_appends_and_steps_store_the_same_keys(gpu, d, bits, fused_norm):
    rng = np.random.default_rng(300 + d + bits)
    B, H, G, n = 2, 2, 4, 150
    cap = n + 64
    tk_bits, tinv = synth.make_transform(H, d, 9, False)
    tk = to_dev_bf16(tk_bits, gpu)
    k = oracle.f32_to_bf16((rng.standard_t(3.0, (B, n, H, d)) * 2.0).astype(np.float32))
    v = oracle.f32_to_bf16(rng.standard_normal((B, n, H, d)).astype(np.float32))
    table = None
    if fused_norm:
        table = torch.from_numpy(synth.rope_table(1e6, d, cap + S_SINK + 64)).to(gpu)
    say("key paths d=%d bits=%d fused norm %s" % (d, bits, fused_norm))

    # one call of n tokens per sequence: the prefill tiles
    c_pre = _cache(gpu, B, H, d, bits, cap)
    kt_pre = _append(c_pre, k, v, [n] * B, tk, table)

    # calls of 13 tokens (the short-append kernel), the last one shorter
    c_short = _cache(gpu, B, H, d, bits, cap)
    kt_short = np.zeros_like(kt_pre)
    for t0 in range(0, n, 13):
        m = min(13, n - t0)
        kt_short[:, t0:t0 + m] = _append(c_short, np.ascontiguousarray(k[:, t0:t0 + m]),
                                         np.ascontiguousarray(v[:, t0:t0 + m]), [m] * B, tk, table)
    assert np.array_equal(kt_short, kt_pre), "k~ of short appends differs from the prefill's"
    _same_state(c_short, c_pre, "short appends vs prefill")

    if fused_norm:
        return
    # fused decode steps (wushkv_decode_step, keys after norm and RoPE): the
    # first 40 tokens by a prefill, the rest one step at a time
    c_step = _cache(gpu, B, H, d, bits, cap)
    _append(c_step, np.ascontiguousarray(k[:, :40]), np.ascontiguousarray(v[:, :40]), [40] * B, tk)
    ones = torch.ones(B, dtype=torch.int32, device=gpu)
    tinv_d = torch.from_numpy(tinv).to(gpu)
    q = to_dev_bf16(oracle.f32_to_bf16(rng.standard_normal((B, H * G, d)).astype(np.float32)), gpu)
    for t in range(40, n):
        wk.wushkv_decode_step(c_step, to_dev_bf16(np.ascontiguousarray(k[:, t]), gpu),
                              to_dev_bf16(np.ascontiguousarray(v[:, t]), gpu), ones, tk, q, tinv_d,
                              sm_scale=1.0 / np.sqrt(d))
    _same_state(c_step, c_pre, "fused steps vs prefill")
    say("  prefill, short appends and fused steps leave identical caches")
