"""The streaming-read reference reads every byte: its per-block XOR equals the
host's XOR of the same bytes, in both load modes."""
import numpy as np
import pytest
import torch

import paper_2609_38121_amd as wk

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("mode", [0, 1])
def test_read_probe_reads_every_word(gpu, mode):
    rng = np.random.default_rng(mode)
    host = rng.integers(0, 2 ** 32, size=(6 * 65536) // 4, dtype=np.uint32)
    buf = torch.from_numpy(host.view(np.int32)).to(gpu)
    sink = wk.wushkv_read_probe(buf, mode)
    torch.cuda.synchronize()
    got = sink.cpu().numpy().view(np.uint32)
    want = np.bitwise_xor.reduce(host.reshape(6, -1), axis=1)
    assert np.array_equal(got, want)
