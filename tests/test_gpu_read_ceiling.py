"""The streaming-read kernel behind the bench's read ceiling reads every
16-byte word of its buffer exactly once: the fold it stores per 64 KiB chunk
(the XOR over the chunk's words of the 32-bit sum of the word's four u32
lanes) matches the same fold computed on the host, chunk by chunk, on sizes
that cover one word, a partial chunk, a ragged last chunk and many chunks;
the sink word past the last chunk is left alone.
"""
from __future__ import annotations

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

CHUNK = 65536


def _folds(words):
    """Per-chunk folds of a uint32 array holding the buffer."""
    lanes = words.reshape(-1, 4).astype(np.uint64)
    sums = (lanes.sum(axis=1) & 0xFFFFFFFF).astype(np.uint32)
    per = CHUNK // 16
    return np.array([np.bitwise_xor.reduce(sums[i:i + per]) for i in range(0, sums.size, per)], np.uint32)


@pytest.mark.parametrize("nbytes", [16, 16 * 255, CHUNK + 48, (3 << 20) + 16])
def test_read_ceiling_reads_every_word_once(nbytes):
    import torch

    import paper_2609_00224_amd as q

    assert torch.cuda.is_available(), "GPU tests need a GPU"
    print(f"[case] read ceiling {nbytes} bytes", flush=True)
    rng = np.random.default_rng(nbytes)
    host = rng.integers(0, 2**32, size=nbytes // 4, dtype=np.uint32)
    buf = torch.from_numpy(host.view(np.uint8).copy()).to("cuda")
    words = q.read_ceiling_sink_words(nbytes)
    assert words == -(-nbytes // CHUNK)
    sink = torch.full((words + 1,), 0x5A5A5A5A, dtype=torch.int32, device="cuda")
    q.qtea_read_ceiling(buf, sink)
    torch.cuda.synchronize()
    got = sink.cpu().numpy().view(np.uint32)
    np.testing.assert_array_equal(got[:words], _folds(host))
    assert got[words] == 0x5A5A5A5A
