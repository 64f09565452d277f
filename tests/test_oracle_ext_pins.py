"""Pins of the oracle's layer-range / prefix swaps and image migration.

* brute force over the 6-D pool index for images with more blocks per layer
  than the table (a cached prefix read from a longer image) and for layer
  subsets (a layer-by-layer offload);
* numpy: take along the block axis, then the layer slice and the first m
  image blocks;
* swapping the layers in groups, one call per group, equals one whole swap;
* migration equals numpy slice assignment; overlaps and bad sizes are
  rejected with no effect.
"""
import itertools

import numpy as np
import pytest

import oracle
from tests.checkers import assert_bytes_equal

EL = {1: np.uint8, 2: np.uint16}


def _rand(rng, n, e):
    return rng.integers(0, 1 << (8 * e), size=n, dtype=np.uint64).astype(EL[e])


@pytest.mark.parametrize("shape", [(2, 6, 1, 2, 4, 2), (3, 5, 1, 1, 8, 2), (3, 8, 1, 2, 8, 1)])
def test_ex_forms_match_brute_force(shape):
    L, N, H, T, D, e = shape
    dt = {1: oracle.FP8_E4M3, 2: oracle.BF16}[e]
    d = oracle.desc(L, N, H, T, D, dt)
    C = oracle.chunk_bytes(d)
    ne = C // e
    rng = np.random.default_rng(400 + N)
    for n in range(0, 3):
        for bt in itertools.permutations(range(N), n):
            for m in (n, n + 2):                # image blocks per layer
                for l0, nl in [(0, 0), (0, 1), (L - 1, 1), (1, L - 1)]:
                    pool = _rand(rng, L * N * 2 * H * T * D, e)
                    img0 = _rand(rng, L * m * ne, e)
                    lay = range(L) if nl == 0 else range(l0, l0 + nl)
                    # swap-out, brute force: every element at its 6-D index
                    img = img0.copy()
                    assert oracle.swap_out_ex(d, pool.view(np.uint8), [list(bt)],
                                              img.view(np.uint8), None, [m], l0, nl) == 0
                    want = img0.copy()
                    for l in lay:
                        for i in range(n):
                            for k in range(ne):
                                want[(l * m + i) * ne + k] = pool[(l * N + bt[i]) * ne + k]
                    assert_bytes_equal(img, want, f"out bt={bt} m={m} l0={l0} nl={nl}")
                    # swap-in, brute force
                    p2 = pool.copy()
                    assert oracle.swap_in_ex(d, p2.view(np.uint8), [list(bt)],
                                             img0.view(np.uint8), None, [m], l0, nl) == 0
                    want = pool.copy()
                    for l in lay:
                        for i in range(n):
                            for k in range(ne):
                                want[(l * N + bt[i]) * ne + k] = img0[(l * m + i) * ne + k]
                    assert_bytes_equal(p2, want, f"in bt={bt} m={m} l0={l0} nl={nl}")


def test_prefix_and_layer_slices_match_numpy():
    rng = np.random.default_rng(410)
    L, N, H, T, D = 4, 32, 2, 4, 8
    d = oracle.desc(L, N, H, T, D, oracle.F16)
    C = oracle.chunk_bytes(d)
    for case in range(300):
        pool = _rand(rng, L * N * 2 * H * T * D, 2)
        p6 = pool.reshape(L, N, 2, H, T, D)
        S = int(rng.integers(1, 4))
        tabs = [list(rng.choice(N, size=int(rng.integers(0, 6)), replace=False)) for _ in range(S)]
        mb = [len(t) + int(rng.integers(0, 3)) for t in tabs]
        l0 = int(rng.integers(0, L))
        nl = int(rng.integers(1, L - l0 + 1))
        size = sum(L * m * C for m in mb)
        img = np.zeros(size, dtype=np.uint8)
        assert oracle.swap_out_ex(d, pool.view(np.uint8), tabs, img, None, mb, l0, nl) == 0
        pos = 0
        for t, m in zip(tabs, mb):
            seg = img[pos:pos + L * m * C].view(np.uint16).reshape(L, m, 2, H, T, D)
            got = seg[l0:l0 + nl, :len(t)]
            want = p6.take(np.asarray(t, dtype=np.int64), axis=1)[l0:l0 + nl]
            assert np.array_equal(got, want), case
            rest = np.concatenate([seg[:l0].reshape(-1), seg[l0 + nl:].reshape(-1),
                                   seg[l0:l0 + nl, len(t):].reshape(-1)])
            assert not rest.any(), case          # nothing else written
            pos += L * m * C


def test_layer_groups_compose_to_a_whole_swap():
    """Swapping in layer groups (one call each) gives the whole swap."""
    rng = np.random.default_rng(420)
    L, N, H, T, D = 6, 40, 1, 4, 8
    d = oracle.desc(L, N, H, T, D, oracle.BF16)
    C = oracle.chunk_bytes(d)
    pool = _rand(rng, L * N * 2 * H * T * D, 2).view(np.uint8)
    bt = [3, 17, 5, 9, 30]
    whole = np.zeros(L * len(bt) * C, dtype=np.uint8)
    assert oracle.swap_out(d, pool, [bt], whole) == 0
    parts = np.zeros_like(whole)
    for l0, nl in [(0, 2), (2, 1), (3, 3)]:
        assert oracle.swap_out_ex(d, pool, [bt], parts, None, None, l0, nl) == 0
    assert_bytes_equal(parts, whole, "layer groups, swap-out")
    bt2 = [0, 1, 2, 38, 39]
    p_whole, p_parts = pool.copy(), pool.copy()
    assert oracle.swap_in(d, p_whole, [bt2], whole) == 0
    for l0, nl in [(0, 1), (1, 4), (5, 1)]:
        assert oracle.swap_in_ex(d, p_parts, [bt2], whole, None, None, l0, nl) == 0
    assert_bytes_equal(p_parts, p_whole, "layer groups, swap-in")


def test_prefix_swap_in_repeated_from_one_cached_image():
    """A long prompt's image is cached once; its first m blocks are swapped
    in repeatedly to fresh blocks and always equal the cached prefix."""
    rng = np.random.default_rng(430)
    L, N, H, T, D = 3, 64, 1, 4, 8
    d = oracle.desc(L, N, H, T, D, oracle.BF16)
    C = oracle.chunk_bytes(d)
    pool = _rand(rng, L * N * 2 * H * T * D, 2).view(np.uint8)
    P = pool.reshape(L, N, C)
    prompt = list(rng.choice(N, size=20, replace=False))
    img = np.zeros(L * 20 * C, dtype=np.uint8)
    assert oracle.swap_out(d, pool, [prompt], img) == 0
    free = [b for b in range(N) if b not in prompt]
    for rep in range(5):
        m = int(rng.integers(1, 21))
        fresh = list(rng.choice(free, size=m, replace=False))
        assert oracle.swap_in_ex(d, pool, [fresh], img, None, [20]) == 0
        assert np.array_equal(P[:, fresh], img.reshape(L, 20, C)[:, :m])


def test_ex_validation():
    L, N = 2, 8
    d = oracle.desc(L, N, 1, 2, 8, oracle.BF16)
    C = oracle.chunk_bytes(d)
    pool = np.zeros(L * N * C, dtype=np.uint8)
    img = np.zeros(L * 4 * C, dtype=np.uint8)
    assert oracle.swap_out_ex(d, pool, [[1, 2]], img, None, [1]) == oracle.ERR_INVALID  # m < n
    assert oracle.swap_out_ex(d, pool, [[1]], img, None, None, 1, 2) == oracle.ERR_INVALID
    assert oracle.swap_out_ex(d, pool, [[1]], img, None, None, 1, 0) == oracle.ERR_INVALID
    assert oracle.swap_in_ex(d, pool, [[1]], img, None, [5]) == oracle.ERR_CAPACITY
    assert oracle.swap_in_ex(d, pool, [[1]], img, None, [4], 1, 1) == 0
    # Placed images whose full extents overlap are rejected even when the
    # layers moved would not touch the overlap.
    assert oracle.swap_out_ex(d, pool, [[1], [2]], img, [0, C], [1, 1], 0, 1) == \
        oracle.ERR_DUPLICATE


def test_migrate_matches_slices_and_rejects_overlaps():
    rng = np.random.default_rng(440)
    src = rng.integers(0, 256, size=4096, dtype=np.uint8)
    dst = rng.integers(0, 256, size=4096, dtype=np.uint8)
    want = dst.copy()
    so, do, ln = [0, 1024, 3072], [2048, 0, 512], [512, 256, 1024]
    for a, b, n in zip(so, do, ln):
        want[b:b + n] = src[a:a + n]
    assert oracle.migrate(src, dst, so, do, ln) == 0
    assert_bytes_equal(dst, want, "migrate")
    d0 = dst.copy()
    assert oracle.migrate(src, dst, [0, 16], [0, 16], [32, 16]) == oracle.ERR_DUPLICATE
    assert oracle.migrate(src, dst, [0], [8], [16]) == oracle.ERR_INVALID
    assert oracle.migrate(src, dst, [0], [0], [24]) == oracle.ERR_INVALID
    assert oracle.migrate(src, dst, [4096 - 16], [0], [32]) == oracle.ERR_CAPACITY
    assert oracle.migrate(src, dst, [0], [4096], [16]) == oracle.ERR_CAPACITY
    # Within one buffer: source and destination ranges must not overlap.
    assert oracle.migrate(dst, dst, [0], [16], [32]) == oracle.ERR_DUPLICATE
    assert_bytes_equal(dst, d0, "failed migrations changed the buffer")
    assert oracle.migrate(dst, dst, [0], [64], [64]) == 0
    assert np.array_equal(dst[64:128], d0[0:64])
