"""The streaming-read measurement hook (kva_debug_stream_read): every word of
the buffer is read, whatever the size and the number of blocks."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("nbytes", [16, 4096 + 48, (1 << 20) + 16 * 37, 64 << 20])
@pytest.mark.parametrize("sink_words", [1, 7, 512, 600])
def test_stream_read_covers_every_word(nbytes, sink_words):
    import torch
    import paper_2609_12471_amd as kva
    print(f"[stream] bytes={nbytes} sink={sink_words}", flush=True)
    rng = np.random.default_rng(nbytes % 1000 + sink_words)
    words = rng.integers(0, 2 ** 32, size=nbytes // 4, dtype=np.uint32)
    src = torch.from_numpy(words.view(np.int32)).cuda()
    sink = torch.zeros(sink_words, dtype=torch.int32, device="cuda")
    kva.kva_debug_stream_read(src, sink)
    torch.cuda.synchronize()
    got = np.bitwise_xor.reduce(sink.cpu().numpy().view(np.uint32))
    assert int(got) == int(np.bitwise_xor.reduce(words))
    if sink_words > 512:
        assert int(sink[512:].count_nonzero()) == 0      # at most 512 blocks
