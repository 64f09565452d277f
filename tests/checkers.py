"""Checkers shared by the oracle pins and the GPU parity tests.

These inspect results; they compute neither side of a swap.
"""
from __future__ import annotations

import numpy as np

_C1 = np.uint64(0xBF58476D1CE4E5B9)
_C2 = np.uint64(0x94D049BB133111EB)


def _mix(z):
    with np.errstate(over="ignore"):
        z = (z ^ (z >> np.uint64(30))) * _C1
        z = (z ^ (z >> np.uint64(27))) * _C2
    return z ^ (z >> np.uint64(31))


def chunk_digests(chunks: np.ndarray) -> np.ndarray:
    """64-bit digest of each row of a [n, C] uint8 array.

    h = C; for every little-endian 8-byte word w of the chunk: h = mix(h ^ w),
    with mix the SplitMix64 finaliser."""
    chunks = np.ascontiguousarray(chunks)
    n, C = chunks.shape
    assert C % 8 == 0
    words = chunks.view("<u8").reshape(n, C // 8)
    h = np.full(n, C, dtype=np.uint64)
    for j in range(C // 8):
        h = _mix(h ^ words[:, j])
    return h


def pool_chunks(pool: np.ndarray, L: int, N: int, C: int) -> np.ndarray:
    """View of a flat uint8 pool as [L, N, C]."""
    return pool[:L * N * C].reshape(L, N, C)


def image_chunks(buf: np.ndarray, off: int, L: int, n: int, C: int) -> np.ndarray:
    """View of one layer-major image [L, n, C] starting at byte ``off``."""
    return buf[off:off + L * n * C].reshape(L, n, C)


def assert_bytes_equal(a: np.ndarray, b: np.ndarray, what: str = "",
                       slab: int = 1 << 28) -> None:
    """Byte-exact comparison that names the first differing offset.  Large
    arrays are compared slab by slab to bound temporary memory."""
    a = np.ascontiguousarray(a).reshape(-1).view(np.uint8)
    b = np.ascontiguousarray(b).reshape(-1).view(np.uint8)
    assert a.size == b.size, f"{what}: size {a.size} != {b.size}"
    for s in range(0, a.size, slab):
        x, y = a[s:s + slab], b[s:s + slab]
        if not np.array_equal(x, y):
            bad = np.flatnonzero(x != y)
            raise AssertionError(
                f"{what}: {bad.size} bytes differ in slab at {s}, first at "
                f"{s + int(bad[0])} ({int(x[bad[0]]):#04x} != {int(y[bad[0]]):#04x})")
