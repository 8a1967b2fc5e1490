"""The plain streaming-read kernel behind the benchmark's bandwidth ceiling
(wici_stream_read): every 32-bit word of the buffer is read exactly once,
checked by the XOR of all words against the host's, for several grids and
sizes (including grids with more workgroups than 16 KiB blocks)."""

from __future__ import annotations

import numpy as np
import pytest

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("mib,grid", [(1, 512), (16, 768), (64, 1024), (3, 7)])
def test_stream_read_touches_every_word_once(cuda_ok, mib, grid):
    import torch

    from paper_2608_24204_amd import binding
    rng = np.random.default_rng(mib * 1000 + grid)
    words = rng.integers(0, 2**32, (mib << 20) // 4, dtype=np.uint64).astype(np.uint32)
    buf = torch.from_numpy(words.view(np.int32)).to("cuda")
    sink = torch.empty(4 * (256 * grid + 1), dtype=torch.uint8, device="cuda")
    ms, ck = binding.stream_read(buf, grid, 2, sink, checksum=True)
    assert ck == int(np.bitwise_xor.reduce(words))
    assert ms > 0


def test_stream_read_rejects_bad_sizes(cuda_ok):
    import torch

    from paper_2608_24204_amd import binding
    buf = torch.zeros(16384 + 4, dtype=torch.uint8, device="cuda")
    sink = torch.empty(4 * (256 * 8 + 1), dtype=torch.uint8, device="cuda")
    with pytest.raises(binding.WiciError) as e:
        binding.stream_read(buf, 8, 1, sink)
    assert e.value.status == binding.WICI_E_ARG
