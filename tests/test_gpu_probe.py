"""hs_stream_read (the streaming-read probe bench.py's read calibration times): every 16-byte
vector is read exactly once, so the XOR of the per-wave words equals the XOR of the buffer's
32-bit words, for every unroll, cache hint and grid, with a ragged tail."""
import numpy as np
import pytest
import torch

import paper_2510_20064_amd as hs

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("unroll", [1, 2, 4, 8])
@pytest.mark.parametrize("nontemporal", [False, True])
@pytest.mark.parametrize("words,grid", [(4, 1), (4 * 1000 + 12, 3), (1 << 20, 64), ((1 << 22) + 36, 517)])
def test_stream_read_reads_every_word_once(unroll, nontemporal, words, grid):
    print("\n[case] unroll=%d nt=%d words=%d grid=%d" % (unroll, nontemporal, words, grid), flush=True)
    rng = np.random.default_rng(words + grid)
    x = rng.integers(-2**31, 2**31, words, dtype=np.int64).astype(np.int32)
    out = hs.stream_read(torch.from_numpy(x).cuda(), grid=grid, unroll=unroll,
                         nontemporal=nontemporal)
    torch.cuda.synchronize()
    got = np.bitwise_xor.reduce(out.cpu().numpy().view(np.uint32))
    assert got == np.bitwise_xor.reduce(x.view(np.uint32))
