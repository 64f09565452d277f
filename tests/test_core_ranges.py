"""The swap space's range allocator against a brute-force model: an array
of unit cells, first fit scanned cell by cell."""
import numpy as np

from tests import core_lib


class Model:
    def __init__(self, size, align):
        self.align = align
        self.cells = np.zeros(size // align, dtype=np.int64)   # 0 free, else owner id
        self.ranges = {}
        self.next = 1

    def alloc(self, nbytes):
        k = -(-nbytes // self.align)
        if nbytes == 0 or k > len(self.cells):
            return None
        run = 0
        for i, c in enumerate(self.cells):
            run = run + 1 if c == 0 else 0
            if run == k:
                lo = i - k + 1
                self.cells[lo:i + 1] = self.next
                self.ranges[lo * self.align] = (k, self.next)
                self.next += 1
                return lo * self.align
        return None

    def free(self, off):
        if off not in self.ranges:
            return False
        k, _ = self.ranges.pop(off)
        self.cells[off // self.align: off // self.align + k] = 0
        return True

    def free_bytes(self):
        return int((self.cells == 0).sum()) * self.align

    def largest_free(self):
        best = run = 0
        for c in self.cells:
            run = run + 1 if c == 0 else 0
            best = max(best, run)
        return best * self.align


def test_first_fit_matches_the_cell_model():
    rng = np.random.default_rng(800)
    for case in range(40):
        align = int(rng.choice([16, 256]))
        size = int(rng.integers(1, 200)) * align + int(rng.integers(0, align))
        r, m = core_lib.Ranges(size, align), Model(size, align)
        live = []
        try:
            for step in range(300):
                if live and rng.random() < 0.45:
                    off = live.pop(int(rng.integers(0, len(live))))
                    assert r.free(off) and m.free(off)
                else:
                    nbytes = int(rng.integers(0, 40 * align))
                    a, b = r.alloc(nbytes), m.alloc(nbytes)
                    assert a == b, (case, step, nbytes)
                    if a is not None:
                        assert a % align == 0 and a + nbytes <= size
                        live.append(a)
                assert r.free_bytes() == m.free_bytes()
                assert r.largest_free() == m.largest_free()
            # Freeing what is not allocated fails and changes nothing.
            fb = r.free_bytes()
            assert not r.free(size + align) and r.free_bytes() == fb
            for off in live:
                assert r.free(off)
                assert not r.free(off)
            assert r.free_bytes() == r.largest_free() == size - size % align
        finally:
            r.close()


def test_coalescing_restores_one_free_range():
    r = core_lib.Ranges(1 << 20, 256)
    try:
        offs = [r.alloc(1000) for _ in range(100)]          # 1024 bytes each
        assert offs == [i * 1024 for i in range(100)]
        for off in offs[::2] + offs[1::2]:                   # free in two interleaved passes
            r.free(off)
        assert r.largest_free() == 1 << 20
        assert r.alloc((1 << 20) + 1) is None and r.alloc(1 << 20) == 0
    finally:
        r.close()
