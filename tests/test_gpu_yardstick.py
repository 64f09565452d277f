"""GPU checks of the HBM yardsticks (aqua_hbm_yardstick): the copy is exact
on a ragged length, the write leaves its documented pattern and nothing
beyond its range, the read writes nothing, and bad arguments are refused
before anything is enqueued."""

import numpy as np
import pytest
import torch

from paper_2407_21255_amd import aqua
from tests.gpu_util import say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    aqua.load()
    yield
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


# 64 MiB plus a ragged tail of 3 vectors: full 64 KiB pieces and one partial.
N = (64 << 20) + 48
GUARD = 4096


def _buffers():
    src = torch.randint(0, 256, (N,), dtype=torch.uint8, device="cuda")
    dst = torch.full((N + 2 * GUARD,), 0xCD, dtype=torch.uint8, device="cuda")
    return src, dst


def test_copy_is_exact():
    src, dst = _buffers()
    s = torch.cuda.Stream()
    aqua.hbm_yardstick(aqua.AQUA_YARDSTICK_COPY, dst[GUARD:GUARD + N], src, stream=s)
    s.synchronize()
    d = dst.cpu().numpy()
    assert np.array_equal(d[GUARD:GUARD + N], src.cpu().numpy())
    assert (d[:GUARD] == 0xCD).all() and (d[GUARD + N:] == 0xCD).all()


def test_write_pattern_and_bounds():
    _, dst = _buffers()
    aqua.hbm_yardstick(aqua.AQUA_YARDSTICK_WRITE, dst[GUARD:GUARD + N])
    torch.cuda.synchronize()
    d = dst.cpu().numpy()
    words = d[GUARD:GUARD + N].view(np.uint32).reshape(-1, 4)
    i = np.arange(N // 16, dtype=np.uint64)
    assert np.array_equal(words[:, 0], (i & 0xFFFFFFFF).astype(np.uint32))
    assert np.array_equal(words[:, 1], (i >> np.uint64(32)).astype(np.uint32))
    assert (words[:, 2] == 0x9E3779B9).all() and (words[:, 3] == 0x61C88646).all()
    assert (d[:GUARD] == 0xCD).all() and (d[GUARD + N:] == 0xCD).all()


def test_read_writes_nothing():
    src, dst = _buffers()
    aqua.hbm_yardstick(aqua.AQUA_YARDSTICK_READ, dst[GUARD:GUARD + 16], src)
    torch.cuda.synchronize()
    assert (dst.cpu().numpy() == 0xCD).all()


def test_bad_arguments_are_refused():
    src, dst = _buffers()
    L = aqua.load()
    d, q = dst.data_ptr() + GUARD, src.data_ptr()
    host = torch.empty(4096, dtype=torch.uint8, pin_memory=True)
    cases = {
        "unknown kind": (3, d, q, 1024),
        "odd length": (0, d, q, 1000),
        "misaligned dst": (0, d + 8, q, 1024),
        "range past the allocation": (0, d, q, 1 << 40),
        "overlapping copy": (0, q + 16, q, 1024),
        "pinned host source": (1, d, host.data_ptr(), 4096),
        "null destination": (2, None, None, 1024),
    }
    for what, (kind, a, b, n) in cases.items():
        st = L.aqua_hbm_yardstick(kind, a, b, n, None)
        say(what, st)
        assert st == aqua.AQUA_ERR_INVALID, what
    assert L.aqua_hbm_yardstick(0, d, q, 0, None) == aqua.AQUA_OK
    torch.cuda.synchronize()
    assert (dst.cpu().numpy() == 0xCD).all()
