"""Choice of the copy engines for the two link directions from the HSA
runtime's availability and preference masks and the set of engines that
carry the host link at its rate (host core, CPU only)."""
import ctypes
import random

import pytest

from tests.core_lib import lib


FAST = 0xF  # engines 0-3


def _pick(av0, pr0, av1, pr1, fast=FAST):
    f = lib().aqua_core_pick_link_engines
    f.argtypes = [ctypes.c_uint32] * 5 + [ctypes.POINTER(ctypes.c_int32)] * 2
    f.restype = None
    d, h = ctypes.c_int32(), ctypes.c_int32()
    f(av0, pr0, av1, pr1, fast, ctypes.byref(d), ctypes.byref(h))
    return d.value, h.value


@pytest.mark.parametrize("masks, want", [
    ((0xFFFF, 0, 0xFFFF, 0), (0, 1)),        # all engines free, no preference: 0 out, 1 in
    ((0xFFFF, 0x4, 0xFFFF, 0x8), (2, 3)),    # preferences honoured
    ((0xFFFF, 0x4, 0xFFFF, 0x4), (2, 2)),    # one preferred engine for both directions
    ((0xFFFC, 0, 0xFFFC, 0), (2, 3)),        # 0 and 1 busy (another pool): the next fast ones
    ((0xFFF0, 0, 0xFFF0, 0), (0, 1)),        # every fast engine busy: share them, not 4+
    ((0xF0, 0x1, 0xF0, 0), (0, 1)),          # preferred and fast engines all busy: share the fast ones
    ((0xFFFE, 0, 0xFFF1, 0), (1, 0)),
    ((0, 0, 0, 0), (0, 1)),                  # nothing reported free: share the fast engines
    ((0x1, 0, 0x1, 0), (0, 0)),              # one free fast engine for both directions
])
def test_fixed_cases(masks, want):
    assert _pick(*masks) == want


def _lowest(m):
    return (m & -m).bit_length() - 1 if m else -1


def _candidates(av, pr, fast):
    if pr & av:
        return pr & av
    f = fast or av
    return (f & av) or f


@pytest.mark.parametrize("fast", [FAST, 0x3, 0])
def test_random_masks_follow_the_rule(fast):
    rng = random.Random(5)
    for _ in range(5000):
        av0, pr0, av1, pr1 = (rng.getrandbits(16) & rng.choice([0xFFFF, 0xFF, 0xF, 0x3, 0])
                              for _ in range(4))
        d2h, h2d = _pick(av0, pr0, av1, pr1, fast)
        # Device to host: the lowest candidate.
        assert d2h == _lowest(_candidates(av0, pr0, fast))
        # Host to device: the same rule, avoiding the device-to-host engine
        # when another candidate exists.
        cand1 = _candidates(av1, pr1, fast)
        if d2h >= 0 and cand1 & ~(1 << d2h):
            cand1 &= ~(1 << d2h)
        assert h2d == _lowest(cand1)
        if fast:
            # Never an engine outside the fast set unless it is preferred.
            assert d2h < 0 or (fast | (pr0 & av0)) >> d2h & 1
            assert h2d < 0 or (fast | (pr1 & av1)) >> h2d & 1
