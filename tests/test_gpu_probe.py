"""The HBM read probe reads every word once: its XOR equals numpy's over the
same bytes, for sizes with and without a tail of the unrolled loop."""
from __future__ import annotations

import numpy as np
import pytest

from paper_2607_14952_amd import binding as B
from tests._gpu import announce

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("n_words", [4, 4 * 2048 * 256 * 8, 4 * 2048 * 256 * 8 * 3 + 4 * 12345])
def test_hbm_read_probe_xor(n_words):
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    rng = np.random.default_rng(n_words)
    host = rng.integers(-2 ** 31, 2 ** 31, size=n_words, dtype=np.int64).astype(np.int32)
    buf = torch.from_numpy(host).cuda()
    announce(f"hbm read probe {n_words * 4} bytes")
    out = B.hbm_read_probe(buf)
    torch.cuda.synchronize()
    assert int(out.cpu()[0]) == int(np.bitwise_xor.reduce(host))
