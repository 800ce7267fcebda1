"""The streaming-read probes read every source word once: the xor of the sink
words is the xor of the source words (computed on the CPU), for one block, for
more threads than words, and for sizes that are not a multiple of the grid's
stride or of a wave's chunk, in every access pattern."""
import numpy as np
import pytest
import torch

import paper_2605_17757_amd as ok

pytestmark = pytest.mark.gpu

CASES = [(1, 1), (1000003, 7), (4096 * 64, 64), (12345, 200)]


@pytest.mark.parametrize("n_words,blocks", CASES)
def test_read_probe_reads_every_word_once(n_words, blocks):
    rng = np.random.default_rng(n_words)
    host = rng.integers(0, 2 ** 32, size=4 * n_words, dtype=np.uint32)  # 16-byte words
    src = torch.from_numpy(host.view(np.int32)).cuda()
    sink = ok.hbm_read_probe(src, blocks)
    torch.cuda.synchronize()
    assert np.bitwise_xor.reduce(sink.cpu().numpy().view(np.uint32)) == np.bitwise_xor.reduce(host)


@pytest.mark.parametrize("loads", [4, 8, 16])
@pytest.mark.parametrize("flags", [0, 1, 2, 3])
@pytest.mark.parametrize("n_words,blocks", CASES)
def test_read_probe_ex_reads_every_word_once(n_words, blocks, loads, flags):
    rng = np.random.default_rng(n_words + 7 * loads + flags)
    host = rng.integers(0, 2 ** 32, size=4 * n_words, dtype=np.uint32)
    src = torch.from_numpy(host.view(np.int32)).cuda()
    sink = ok.hbm_read_probe(src, blocks, loads=loads, flags=flags)
    torch.cuda.synchronize()
    assert np.bitwise_xor.reduce(sink.cpu().numpy().view(np.uint32)) == np.bitwise_xor.reduce(host)
