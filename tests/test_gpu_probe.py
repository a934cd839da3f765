"""The streaming-read probe (a measurement aid, no part of the method): its per-workgroup
sums of 32-bit words add up, with wrapping, to the sum of every word of the buffer."""
import numpy as np
import pytest
import torch

import paper_2606_24957_amd as D

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _wrapping_sum(words: np.ndarray) -> int:
    return int(words.astype(np.uint64).sum() % (1 << 32))


@pytest.mark.parametrize("n_words,blocks", [(4, 1), (4096, 7), (1 << 20, 1024), (3 * (1 << 18) + 12, 300)])
def test_read_probe_sums(n_words, blocks):
    rng = np.random.default_rng(n_words + blocks)
    words = rng.integers(0, 1 << 32, n_words, dtype=np.uint64).astype(np.uint32)
    data = torch.from_numpy(words.view(np.int32)).to(DEV)
    sums = D.plan_read_probe(data, blocks=blocks)()
    torch.cuda.synchronize()
    got = _wrapping_sum(sums.cpu().numpy().view(np.uint32))
    assert got == _wrapping_sum(words)
    # the runs split the buffer: each workgroup's sum is that of its own run
    per = -(-n_words // 4 // blocks) * 4
    ref = [_wrapping_sum(words[g * per:(g + 1) * per]) for g in range(blocks)]
    assert sums.cpu().numpy().view(np.uint32).tolist() == ref
