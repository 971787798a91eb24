"""The no-allocation decode entry point, wushkv_decode_attention_noalloc (for
callers that cannot allocate device memory), through the C ABI: two calls in
a row, the second on a smaller cache, each against wushkv_decode_attention
with a workspace of its own (the same kernels and plan: identical outputs)
and against the oracle on the GPU's own cache (the row-normalised 2e-3 bar
of the decode parity tests).  It must pass alone in a fresh process and
after the other GPU tests."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_38121_amd as wk
from paper_2609_38121_amd import _lib
from gpu_harness import Pair, TOL, rel_err, say, to_dev_bf16

pytestmark = pytest.mark.gpu


def _kv(rng, B, n, H, d):
    k = rng.standard_normal((B, n, H, d)).astype(np.float32)
    k[..., [5, 40]] *= 8.0
    v = rng.standard_normal((B, n, H, d)).astype(np.float32)
    return oracle.f32_to_bf16(k), oracle.f32_to_bf16(v)


def test_noalloc_decode_matches_the_workspace_call(gpu):
    rng = np.random.default_rng(500)
    cases = [  # (batch, kv heads, G, d, bits, lengths): the second call is smaller
        (4, 4, 4, 128, 2, [3000, 1200, 0, 2500]),
        (2, 2, 2, 64, 4, [700, 90]),
    ]
    for B, H, G, d, bits, lens in cases:
        say("noalloc decode: batch %d, %d kv heads, G %d, d %d, %d-bit, lengths %s" % (B, H, G, d, bits, lens))
        p = Pair(gpu, B, H, G, d, bits, 4, 128, 8, 0.96, 0.92, cap=max(lens) + 64, oracle_ref=False)
        k, v = _kv(rng, B, max(lens), H, d)
        p.append(k, v, lens)
        q = oracle.f32_to_bf16(rng.standard_normal((B, H * G, d)).astype(np.float32))
        qd = to_dev_bf16(q, gpu)
        need = wk.wushkv_decode_workspace_bytes(p.gpu, H * G, p.gpu.max_seq_len)
        assert 0 < need <= _lib.NOALLOC_SCRATCH_BYTES
        ref = wk.wushkv_decode_attention(p.gpu, qd, p.tinv_dev, sm_scale=p.sm_scale)
        out = torch.full((B, H * G, d), float("nan"), dtype=torch.float32, device=gpu)
        wk.wushkv_decode_attention_noalloc(p.gpu, qd, p.tinv_dev, out, sm_scale=p.sm_scale)
        torch.cuda.synchronize()
        got, exp = out.cpu().numpy(), ref.cpu().numpy()
        assert np.all(np.isfinite(got))
        assert np.array_equal(got, exp), "noalloc differs from the workspace call: %.3e" % rel_err(got, exp)
        e = rel_err(got, p.mirror.decode(q, p.tinv, p.sm_scale))
        say("  identical to the workspace call; rel err vs oracle %.2e" % e)
        assert e <= TOL


def test_noalloc_refuses_plans_beyond_its_array(gpu):
    # 256 sequences x 8 kv heads x 8 query heads at 65536 tokens: the split
    # partials alone need far more than the static array holds
    import ctypes
    c = wk.WushKVCache(256, 8, 128, 2, 4, 128, 8, 0.96, 0.92, max_seq_len=256, device=gpu)
    need = wk.wushkv_decode_workspace_bytes(c, 64, 65536)
    assert need > _lib.NOALLOC_SCRATCH_BYTES
    q = torch.zeros(256, 64, 128, dtype=torch.bfloat16, device=gpu)
    out = torch.zeros(256, 64, 128, dtype=torch.float32, device=gpu)
    tinv = torch.zeros(8, 128, 128, dtype=torch.float32, device=gpu)
    st = _lib.lib().wushkv_decode_attention_noalloc(ctypes.byref(c.desc), q.data_ptr(), 64, 65536,
                                                    tinv.data_ptr(), 0.1, out.data_ptr(), None)
    assert st == _lib.EWORKSPACE
