"""Pins of the CPU oracle against facts fixed outside it.

* brute force: an element-by-element loop over the 6-D pool index
  (layer, block, K|V, head, token, dim) with its own row-major strides;
* a library routine: numpy ``take`` / fancy assignment along the block axis;
* round-trip identity, per-chunk digest preservation, guard bands;
* the error table;
* KV sizes printed in the paper and fixed by public model shapes.
"""
import itertools
import json
import os

import numpy as np
import pytest

import oracle
from paper_2407_21255_amd import workload as wl
from tests.checkers import assert_bytes_equal, chunk_digests

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
EL = {1: np.uint8, 2: np.uint16}


def _shape6(L, N, H, T, D):
    return (L, N, 2, H, T, D)


def _random_pool(rng, L, N, H, T, D, e):
    n = L * N * 2 * H * T * D
    return rng.integers(0, 1 << (8 * e), size=n, dtype=np.uint64).astype(EL[e])


def _brute_image(pool_el, shape6, bt):
    """Image elements by an explicit loop over the 6-D index."""
    L, N, KV, H, T, D = shape6
    # Row-major strides of [L][N][2][H][T][D], in elements.
    sd = 1
    st = D
    sh = T * D
    skv = H * T * D
    sb = KV * H * T * D
    sl = N * KV * H * T * D
    n = len(bt)
    img = np.zeros(L * n * KV * H * T * D, dtype=pool_el.dtype)
    pos = 0
    for l in range(L):
        for i in range(n):
            for kv in range(KV):
                for h in range(H):
                    for t in range(T):
                        for d in range(D):
                            img[pos] = pool_el[l * sl + bt[i] * sb + kv * skv +
                                               h * sh + t * st + d * sd]
                            pos += 1
    return img


# (L, N, H, T, D, e) with a chunk size that is a multiple of 16 bytes.
TINY_SHAPES = [(1, 4, 1, 1, 8, 1), (2, 5, 1, 2, 4, 1), (3, 8, 1, 4, 8, 2),
               (2, 8, 1, 1, 4, 2), (3, 6, 1, 2, 8, 1)]


@pytest.mark.parametrize("shape", TINY_SHAPES)
def test_swap_out_matches_brute_force_every_short_table(shape):
    L, N, H, T, D, e = shape
    rng = np.random.default_rng(100 + N)
    pool = _random_pool(rng, L, N, H, T, D, e)
    d = oracle.desc(L, N, H, T, D, {1: oracle.FP8_E4M3, 2: oracle.BF16}[e])
    C = oracle.chunk_bytes(d)
    for n in range(0, 4):
        for bt in itertools.product(range(N), repeat=n):
            img = np.full(L * n * C, 0x5A, dtype=np.uint8)
            assert oracle.swap_out(d, pool.view(np.uint8), [list(bt)], img) == 0
            expect = _brute_image(pool, _shape6(L, N, H, T, D), bt)
            assert_bytes_equal(img, expect.view(np.uint8), f"bt={bt}")


@pytest.mark.parametrize("shape", TINY_SHAPES)
def test_swap_in_matches_brute_force_every_short_table(shape):
    L, N, H, T, D, e = shape
    rng = np.random.default_rng(200 + N)
    d = oracle.desc(L, N, H, T, D, {1: oracle.FP8_E4M3, 2: oracle.BF16}[e])
    C = oracle.chunk_bytes(d)
    ne = C // e
    for n in range(0, 4):
        for bt in itertools.permutations(range(N), n):
            pool = _random_pool(rng, L, N, H, T, D, e)
            img = rng.integers(0, 1 << (8 * e), size=L * n * ne,
                               dtype=np.uint64).astype(EL[e])
            out = pool.copy()
            assert oracle.swap_in(d, out.view(np.uint8), [list(bt)],
                                  img.view(np.uint8)) == 0
            # Brute force: write every image element at its 6-D pool index.
            expect = pool.copy()
            pos = 0
            for l in range(L):
                for i in range(n):
                    for kv in range(2):
                        for h in range(H):
                            for t in range(T):
                                for dd in range(D):
                                    expect[(((((l * N + bt[i]) * 2 + kv) * H + h)
                                             * T + t) * D + dd)] = img[pos]
                                    pos += 1
            assert_bytes_equal(out, expect, f"bt={bt}")


def test_random_multi_sequence_cases_match_numpy_take_and_put():
    """10^4 random calls: numpy take/put along the block axis of the 6-D pool."""
    rng = np.random.default_rng(300)
    for case in range(10_000):
        L = int(rng.integers(1, 4))
        N = int(rng.integers(1, 9))
        H = 1
        T = int(rng.choice([1, 2, 4]))
        D = int(rng.choice([4, 8]))
        e = int(rng.choice([1, 2]))
        if (2 * H * T * D * e) % 16:
            continue
        d = oracle.desc(L, N, H, T, D, {1: oracle.FP8_E4M3, 2: oracle.F16}[e])
        C = oracle.chunk_bytes(d)
        pool = _random_pool(rng, L, N, H, T, D, e)
        p6 = pool.reshape(_shape6(L, N, H, T, D))
        S = int(rng.integers(0, 4))
        out_tables = [list(rng.integers(0, N, size=int(rng.integers(0, 4))))
                      for _ in range(S)]
        total = sum(len(t) for t in out_tables)
        img = np.zeros(L * total * C, dtype=np.uint8)
        assert oracle.swap_out(d, pool.view(np.uint8), out_tables, img) == 0
        pos = 0
        for t in out_tables:
            n = len(t)
            seg = img[pos:pos + L * n * C].view(pool.dtype).reshape(
                (L, n, 2, H, T, D))
            assert np.array_equal(seg, p6.take(np.asarray(t, dtype=np.int64),
                                               axis=1)), case
            pos += L * n * C
        # Swap-in of the same images into distinct blocks.
        perm = rng.permutation(N)
        in_tables, k = [], 0
        for t in out_tables:
            n = min(len(t), N - k)
            in_tables.append([int(x) for x in perm[k:k + n]])
            k += n
        if any(len(a) != len(b) for a, b in zip(in_tables, out_tables)):
            continue
        pool2 = pool.copy()
        assert oracle.swap_in(d, pool2.view(np.uint8), in_tables, img) == 0
        expect = p6.copy()
        pos = 0
        for t in in_tables:
            n = len(t)
            seg = img[pos:pos + L * n * C].view(pool.dtype).reshape(
                (L, n, 2, H, T, D))
            if n:
                expect[:, np.asarray(t, dtype=np.int64)] = seg
            pos += L * n * C
        assert np.array_equal(pool2.reshape(expect.shape), expect), case


def _tiny_pool(case):
    shape = case.shape
    import torch
    pool = torch.empty(shape.pool_bytes, dtype=torch.uint8)
    wl.fill_pool(pool, shape, case.seed, case.owner)
    return pool.numpy()


def test_round_trip_digests_guards_tiny_config():
    """Round trip on the 4-layer fp16 pool: pool'[:, bt2] == pool[:, bt],
    every other chunk unchanged, digests preserved, guards intact, and
    swap-out of bt2 reproduces the first image."""
    case = wl.tiny_case()
    s = case.shape
    d = oracle.desc(*s.as_tuple())
    C = s.chunk_bytes
    pool = _tiny_pool(case)
    bt, bt2 = case.out_tables[0], case.in_tables[0]
    # The destination chunks carry a sentinel so that a missed write shows.
    P = pool.reshape(s.num_layers, s.num_blocks, C)
    P[:, bt2] = wl.SENTINEL_BYTE
    before = pool.copy()
    guard = 4096
    buf = np.full(guard + s.image_bytes(len(bt)) + guard, wl.GUARD_BYTE,
                  dtype=np.uint8)
    assert oracle.swap_out(d, pool, [bt], buf, [guard]) == 0
    assert_bytes_equal(pool, before, "swap-out modified the pool")
    img = buf[guard:guard + s.image_bytes(len(bt))].reshape(s.num_layers, len(bt), C)
    assert np.all(buf[:guard] == wl.GUARD_BYTE) and np.all(buf[-guard:] == wl.GUARD_BYTE)
    assert oracle.swap_in(d, pool, [bt2], buf, [guard]) == 0
    P2 = pool.reshape(s.num_layers, s.num_blocks, C)
    B = before.reshape(s.num_layers, s.num_blocks, C)
    assert np.array_equal(P2[:, bt2], B[:, bt])
    untouched = np.setdiff1d(np.arange(s.num_blocks), bt2)
    assert np.array_equal(P2[:, untouched], B[:, untouched])
    dg_src = chunk_digests(B[:, bt].reshape(-1, C))
    dg_img = chunk_digests(img.reshape(-1, C))
    dg_dst = chunk_digests(P2[:, bt2].reshape(-1, C))
    assert np.array_equal(dg_src, dg_img) and np.array_equal(dg_img, dg_dst)
    assert len(set(dg_src.tolist())) == dg_src.size  # chunks are distinct
    buf2 = np.full_like(buf, wl.GUARD_BYTE)
    assert oracle.swap_out(d, pool, [bt2], buf2, [guard]) == 0
    assert_bytes_equal(buf2, buf, "second swap-out image")


def test_digest_detects_single_byte_change():
    rng = np.random.default_rng(7)
    x = rng.integers(0, 256, size=(4, 64), dtype=np.uint8)
    d0 = chunk_digests(x)
    for pos in [0, 7, 8, 63]:
        y = x.copy()
        y[2, pos] ^= 1
        d1 = chunk_digests(y)
        assert d1[2] != d0[2] and np.array_equal(np.delete(d1, 2), np.delete(d0, 2))


def test_explicit_image_offsets_and_packed_layout():
    """Packed images sit one after another (sequence s at the sum of the
    earlier images' sizes); explicit offsets place each image anywhere."""
    rng = np.random.default_rng(11)
    L, N, H, T, D = 2, 16, 1, 2, 8
    d = oracle.desc(L, N, H, T, D, oracle.F16)
    C = oracle.chunk_bytes(d)
    pool = _random_pool(rng, L, N, H, T, D, 2).view(np.uint8)
    tables = [[3, 4, 5], [], [9], [0, 15]]
    packed = np.zeros(L * 6 * C, dtype=np.uint8)
    assert oracle.swap_out(d, pool, tables, packed) == 0
    offs = [10 * C * L, 0, 3 * C * L, 6 * C * L]
    placed = np.zeros(16 * C * L, dtype=np.uint8)
    assert oracle.swap_out(d, pool, tables, placed, offs) == 0
    pos = 0
    for t, o in zip(tables, offs):
        n = len(t)
        assert_bytes_equal(placed[o:o + L * n * C], packed[pos:pos + L * n * C])
        one = np.zeros(L * n * C, dtype=np.uint8)
        assert oracle.swap_out(d, pool, [t], one) == 0
        assert_bytes_equal(one, packed[pos:pos + L * n * C])
        pos += L * n * C


def test_error_table_and_no_side_effects():
    rng = np.random.default_rng(12)
    L, N, H, T, D = 2, 8, 1, 2, 8
    d = oracle.desc(L, N, H, T, D, oracle.BF16)
    C = oracle.chunk_bytes(d)
    pool = _random_pool(rng, L, N, H, T, D, 2).view(np.uint8)
    img = np.zeros(L * 4 * C, dtype=np.uint8)
    p0, i0 = pool.copy(), img.copy()

    def unchanged():
        assert_bytes_equal(pool, p0, "pool changed by a failing call")
        assert_bytes_equal(img, i0, "image changed by a failing call")

    # Range: negative and >= N.
    assert oracle.swap_out(d, pool, [[0, -1]], img) == oracle.ERR_RANGE
    assert oracle.swap_in(d, pool, [[0, N]], img) == oracle.ERR_RANGE
    # Duplicate destination in one swap-in (also across sequences).
    assert oracle.swap_in(d, pool, [[1, 2], [2]], img) == oracle.ERR_DUPLICATE
    # A swap-out may read one block twice.
    assert oracle.swap_out(d, pool, [[1, 1]], img) == 0
    i0 = img.copy()
    # Overlapping image ranges in one swap-out.
    assert oracle.swap_out(d, pool, [[1], [2]], img, [0, C]) == oracle.ERR_DUPLICATE
    # Capacity.
    assert oracle.swap_out(d, pool, [[1, 2, 3, 4, 5]], img) == oracle.ERR_CAPACITY
    assert oracle.swap_in(d, pool, [[1]], img, [img.nbytes - C]) == oracle.ERR_CAPACITY
    # Misaligned image offset.
    assert oracle.swap_out(d, pool, [[1]], img, [8]) == oracle.ERR_INVALID
    # Bad shape: chunk not a multiple of 16 bytes, zero layers, bad dtype.
    assert oracle.swap_out(oracle.desc(L, N, H, 1, 4, oracle.FP8_E4M3), pool,
                           [[1]], img) == oracle.ERR_INVALID
    assert oracle.swap_out(oracle.desc(0, N, H, T, D, oracle.BF16), pool,
                           [[1]], img) == oracle.ERR_INVALID
    assert oracle.swap_out(oracle.desc(L, N, H, T, D, 9), pool, [[1]],
                           img) == oracle.ERR_INVALID
    # Pool smaller than the shape.
    assert oracle.pool_check(d, pool, pool.nbytes - 1) == oracle.ERR_CAPACITY
    # Precedence: invalid before range before duplicate before capacity.
    assert oracle.swap_in(d, pool, [[N, N]], img, [8]) == oracle.ERR_INVALID
    assert oracle.swap_in(d, pool, [[N, 1, 1]], img) == oracle.ERR_RANGE
    assert oracle.swap_in(d, pool, [[1, 1, 2, 3, 4]], img) == oracle.ERR_DUPLICATE
    unchanged()
    # Empty calls are no-ops.
    assert oracle.swap_out(d, pool, [], img) == 0
    assert oracle.swap_in(d, pool, [[], []], img) == 0
    unchanged()


def test_null_and_offsets_validation():
    import ctypes
    L, N, H, T, D = 1, 4, 1, 1, 8
    d = oracle.desc(L, N, H, T, D, oracle.FP8_E4M3)
    pool = np.zeros(L * N * 16, dtype=np.uint8)
    img = np.zeros(64, dtype=np.uint8)
    lib = oracle.lib()
    ids = np.array([0, 1], dtype=np.int32)
    offs = np.array([0, 2], dtype=np.uint64)
    bad = np.array([1, 2], dtype=np.uint64)
    dec = np.array([0, 2, 1], dtype=np.uint64)
    R = lambda *a: lib.oracle_swap_out(ctypes.byref(d), *a)
    assert R(pool.ctypes.data, pool.nbytes, 1, ids.ctypes.data,
             offs.ctypes.data, img.ctypes.data, img.nbytes, None) == 0
    assert R(None, pool.nbytes, 1, ids.ctypes.data, offs.ctypes.data,
             img.ctypes.data, img.nbytes, None) == oracle.ERR_INVALID
    assert R(pool.ctypes.data, pool.nbytes, 1, None, offs.ctypes.data,
             img.ctypes.data, img.nbytes, None) == oracle.ERR_INVALID
    assert R(pool.ctypes.data, pool.nbytes, 1, ids.ctypes.data, None,
             img.ctypes.data, img.nbytes, None) == oracle.ERR_INVALID
    assert R(pool.ctypes.data, pool.nbytes, 1, ids.ctypes.data,
             offs.ctypes.data, None, img.nbytes, None) == oracle.ERR_INVALID
    assert R(pool.ctypes.data, pool.nbytes, 1, ids.ctypes.data,
             bad.ctypes.data, img.ctypes.data, img.nbytes, None) == oracle.ERR_INVALID
    assert R(pool.ctypes.data, pool.nbytes, 2, ids.ctypes.data,
             dec.ctypes.data, img.ctypes.data, img.nbytes, None) == oracle.ERR_INVALID
    assert R(pool.ctypes.data + 8, pool.nbytes, 1, ids.ctypes.data,
             offs.ctypes.data, img.ctypes.data, img.nbytes, None) == oracle.ERR_INVALID


def test_kv_sizes_against_paper_and_public_shapes():
    dt = {"f16": oracle.F16, "bf16": oracle.BF16}
    with open(os.path.join(GOLDEN, "kv_sizing.json")) as f:
        entries = json.load(f)["entries"]
    for e in entries:
        sh = e["shape"]
        d = oracle.desc(sh["num_layers"], 1, sh["num_kv_heads"], 16,
                        sh["head_dim"], dt[sh["dtype"]])
        got = oracle.bytes_per_token(d) * e["tokens"]
        if "expected_bytes" in e:
            assert got == e["expected_bytes"], e["model"]
        else:
            rel = abs(got - e["expected_bytes_approx"]) / e["expected_bytes_approx"]
            assert rel <= e["tolerance_rel"], (e["model"], got)
    # The chunk is a whole block of K and V for all heads of one layer.
    d = oracle.desc(32, 16384, 8, 16, 128, oracle.BF16)
    assert oracle.chunk_bytes(d) == 64 * 1024
    assert oracle.chunk_bytes(oracle.desc(32, 1, 8, 16, 128, oracle.FP8_E4M3)) == 32 * 1024
    assert oracle.bytes_per_token(d) * 16 == 32 * oracle.chunk_bytes(d)
