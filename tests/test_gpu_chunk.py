"""GPU parity of chunk attention (Alg. 2 step 5 with S' > 1: the causal mask
of Eq. (2) inside each sequence's chunk of new tokens) against the oracle,
on the mirror cache (the GPU's own codes) and the end-to-end reference (with
the GPU's k~ at any position whose codes sit on the other side of a rounding
tie, see gpu_harness.tie_patched)."""
import numpy as np
import pytest
import torch

from gpu_harness import Pair, rel_err, say, to_dev_bf16, TOL
import oracle
import paper_2609_38121_amd as wk

pytestmark = pytest.mark.gpu


def _kv(rng, B, n, H, d):
    k = rng.standard_normal((B, n, H, d)).astype(np.float32)
    v = rng.standard_normal((B, n, H, d)).astype(np.float32)
    return oracle.f32_to_bf16(k), oracle.f32_to_bf16(v)


def _chunk(p, q, n_tok, max_seq_len=None):
    nd = torch.from_numpy(np.asarray(n_tok, np.int32)).to(p.dev)
    out = wk.wushkv_chunk_attention(p.gpu, to_dev_bf16(q, p.dev), p.tinv_dev, n_tok=nd,
                                    sm_scale=p.sm_scale, max_seq_len=max_seq_len)
    torch.cuda.synchronize()
    return out.cpu().numpy()


def _check(p, q, n_tok, max_seq_len=None):
    gpu = _chunk(p, q, n_tok, max_seq_len)
    assert np.all(np.isfinite(gpu))
    mir = oracle.chunk_attention(p.mirror, q, n_tok, p.tinv, p.sm_scale)
    valid = ~np.isnan(mir[..., 0])
    # rows beyond a sequence's chunk are zero
    assert np.all(gpu[~valid] == 0)
    em = rel_err(gpu[valid], mir[valid])
    # the end-to-end reference; where its key codes differ from the GPU's at
    # a rounding tie of k~, the same reference with the GPU's k~ at exactly
    # those positions
    ref, n_sub = p.reference_for(lambda c: oracle.chunk_attention(c, q, n_tok, p.tinv, p.sm_scale))
    er = rel_err(gpu[valid], ref[valid])
    say("  chunk rel err vs mirror %.2e, vs reference %.2e (%d tie positions substituted)"
        % (em, er, n_sub))
    assert em <= TOL
    assert er <= TOL
    return gpu


@pytest.mark.parametrize("d,bits,G", [(128, 2, 4), (128, 4, 8), (128, 3, 2), (64, 2, 1), (64, 4, 2)])
def test_chunk_attention_ragged(gpu, d, bits, G):
    rng = np.random.default_rng(200 + d + bits + G)
    B, H, T = 3, 2, 16
    say("chunk d=%d bits=%d G=%d" % (d, bits, G))
    p = Pair(gpu, B, H, G, d, bits, 4, 128, 8, 0.96, 0.92, cap=900, symmetric=False, seed=4)
    k, v = _kv(rng, B, 700, H, d)
    p.append(k, v, [700, 333, 0])
    n_tok = np.array([16, 5, 11])  # the last sequence's chunk is its whole content
    k, v = _kv(rng, B, T, H, d)
    p.append(k, v, n_tok)
    p.check_cache()
    q = oracle.f32_to_bf16(rng.standard_normal((B, T, H * G, d)).astype(np.float32))
    _check(p, q, n_tok)
    # a second chunk on top (crosses a flush)
    n_tok = np.array([9, 16, 2])
    k, v = _kv(rng, B, T, H, d)
    p.append(k, v, n_tok)
    p.check_cache()
    q = oracle.f32_to_bf16(rng.standard_normal((B, T, H * G, d)).astype(np.float32))
    _check(p, q, n_tok)


def test_chunk_of_one_token_is_decode(gpu):
    rng = np.random.default_rng(21)
    B, H, G, d = 2, 2, 4, 128
    p = Pair(gpu, B, H, G, d, 2, 4, 128, 8, 0.96, 0.92, cap=600, oracle_ref=False)
    k, v = _kv(rng, B, 500, H, d)
    p.append(k, v, [500, 260])
    q = oracle.f32_to_bf16(rng.standard_normal((B, 1, H * G, d)).astype(np.float32))
    a = _chunk(p, q, [1, 1])
    b = p.decode(np.ascontiguousarray(q[:, 0]))
    assert np.array_equal(a[:, 0], b)


def test_chunk_at_sequence_start_and_null_counts(gpu):
    """A chunk that is a sequence's whole content (positions from 0, so the
    sink slots past a token's own position are masked too), with n_tok
    omitted (every sequence takes max_tok tokens)."""
    rng = np.random.default_rng(22)
    B, H, G, d, T = 2, 1, 4, 64, 12
    p = Pair(gpu, B, H, G, d, 2, 4, 16, 8, 0.96, 0.92, cap=64)
    k, v = _kv(rng, B, T, H, d)
    p.append(k, v, [T, T])
    q = oracle.f32_to_bf16(rng.standard_normal((B, T, H * G, d)).astype(np.float32))
    gpu_out = wk.wushkv_chunk_attention(p.gpu, to_dev_bf16(q, p.dev), p.tinv_dev,
                                        sm_scale=p.sm_scale)
    torch.cuda.synchronize()
    gpu_out = gpu_out.cpu().numpy()
    ref = oracle.chunk_attention(p.mirror, q, [T, T], p.tinv, p.sm_scale)
    e = rel_err(gpu_out, ref)
    say("  chunk from position 0: rel err %.2e" % e)
    assert e <= TOL
    # token 0 attends to position 0 only: its output is that value row
    v0 = oracle.bf16_to_f32(v[:, 0, 0]).astype(np.float64)
    assert np.allclose(gpu_out[:, 0, :, :], v0[:, None, :], rtol=1e-5, atol=1e-6)


@pytest.mark.timeout(600)
def test_chunk_llama_shaped(gpu):
    """Batch 8, 32 q / 8 kv heads, d 128, 2-bit, 2048-token context, then a
    16-token chunk per sequence: every head against the oracle."""
    rng = np.random.default_rng(23)
    B, H, G, d, T = 8, 8, 4, 128, 16
    p = Pair(gpu, B, H, G, d, 2, 4, 128, 8, 0.96, 0.92, cap=2100, oracle_ref=False)
    k, v = _kv(rng, B, 2048, H, d)
    p.append(k, v, [2048] * B)
    k, v = _kv(rng, B, T, H, d)
    n_tok = np.array([T] * B)
    p.append(k, v, n_tok)
    q = oracle.f32_to_bf16(rng.standard_normal((B, T, H * G, d)).astype(np.float32))
    gpu_out = _chunk(p, q, n_tok)
    mir = oracle.chunk_attention(p.mirror, q, n_tok, p.tinv, p.sm_scale)
    e = rel_err(gpu_out, mir)
    say("  llama-shaped 16-token chunk: rel err %.2e over %d rows" % (e, B * T * H * G))
    assert e <= TOL
