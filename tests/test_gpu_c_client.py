"""The C ABI from a plain C program (tests/c_abi_client.c, built by
build()): no Python or torch in that process.  The program writes the pool
it filled, the images its swap-outs made and the pool after its swap-in;
each is compared byte for byte with the oracle on the same input."""
import os
import subprocess

import numpy as np
import pytest

import oracle
from paper_2407_21255_amd import workload as wl
from tests.checkers import assert_bytes_equal
from tests.gpu_util import say

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CLIENT = os.path.join(ROOT, "tests", "c_abi_client")

# The program's fixed shape and tables.
SHAPE = (4, 64, 8, 16, 128, wl.F16)
OUT = [[5, 9, 10, 11, 40, 2, 63, 0, 33, 34], [7, 8, 20, 61, 62, 1, 3]]
IN = [list(range(41, 51)), list(range(51, 58))]


@pytest.mark.gpu
def test_c_program_swaps_through_the_abi(tmp_path):
    assert os.path.exists(CLIENT), "build() compiles tests/c_abi_client"
    say("c_abi_client", tmp_path)
    r = subprocess.run([CLIENT, str(tmp_path)], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr
    assert r.stdout.strip().endswith("c_abi_client: ok")

    def load(name):
        return np.fromfile(tmp_path / name, dtype=np.uint8)

    pool = load("pool_before.bin")
    assert len(np.unique(pool)) == 256
    d = oracle.desc(*SHAPE)
    img = np.zeros(load("image_hbm.bin").size, dtype=np.uint8)
    assert oracle.swap_out(d, pool.copy(), OUT, img) == 0
    assert_bytes_equal(load("image_hbm.bin"), img, "HBM image")
    assert_bytes_equal(load("image_host.bin"), img, "host image")
    assert oracle.swap_in(d, pool, IN, img) == 0
    assert_bytes_equal(load("pool_after.bin"), pool, "pool after swap-in")
