"""wici_stream_read_noalloc: the streaming-read diagnostic with its workspace in
the library's file-scope device array (for callers that cannot allocate device
memory), checked through the C ABI against wici_stream_read, whose workspace the
caller passes, and against the host's XOR of the buffer.  Two calls in a row,
the second on a smaller buffer with a smaller grid, so a stale larger workspace
would show; a grid beyond the array is rejected."""

from __future__ import annotations

import ctypes

import numpy as np
import pytest

pytestmark = pytest.mark.gpu


def _noalloc(lib, buf, grid):
    import torch
    ck = ctypes.c_uint32()
    st = torch.cuda.current_stream().cuda_stream
    r = lib.wici_stream_read_noalloc(ctypes.c_void_p(buf.data_ptr()),
                                     buf.numel() * buf.element_size(), grid,
                                     ctypes.c_void_p(st), ctypes.byref(ck))
    return r, int(ck.value)


def test_no_alloc_stream_read_matches_the_workspace_call(cuda_ok):
    import torch

    from paper_2608_24204_amd import binding
    lib = binding.load_library()
    for mib, grid in ((64, 1024), (1, 100)):
        rng = np.random.default_rng(mib)
        words = rng.integers(0, 2**32, (mib << 20) // 4, dtype=np.uint64).astype(np.uint32)
        buf = torch.from_numpy(words.view(np.int32)).to("cuda")
        sink = torch.empty(4 * (256 * grid + 1), dtype=torch.uint8, device="cuda")
        r, ck = _noalloc(lib, buf, grid)
        assert r == binding.WICI_OK
        _, ref = binding.stream_read(buf, grid, 1, sink, checksum=True)
        assert ck == ref == int(np.bitwise_xor.reduce(words)), (mib, grid)


def test_no_alloc_stream_read_rejects_a_grid_beyond_its_array(cuda_ok):
    import torch

    from paper_2608_24204_amd import binding
    lib = binding.load_library()
    buf = torch.zeros(1 << 20, dtype=torch.uint8, device="cuda")
    assert _noalloc(lib, buf, 4097)[0] == binding.WICI_E_ARG
    assert _noalloc(lib, buf, 4096)[0] == binding.WICI_OK
