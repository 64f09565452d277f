"""bench.py's host logic, without a GPU: the one-GPU guard, argument
checks, the garbage-collector pause around timed regions and the CPU
baseline record."""
import gc
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
BENCH = os.path.join(ROOT, "bench.py")


def _run(args, env_extra=None):
    env = dict(os.environ)
    env.update(env_extra or {})
    return subprocess.run([sys.executable, BENCH, *args], capture_output=True, text=True,
                          timeout=300, env=env)


def test_more_than_one_gpu_is_refused_with_a_message():
    r = _run(["--gpus", "2"])
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""
    r = _run([], {"WORLD_SIZE": "4"})
    assert r.returncode == 2 and "one GPU" in r.stderr


def test_bad_link_engine_is_an_argument_error():
    r = _run(["--link-engine", "16"])
    assert r.returncode == 2 and "--link-engine" in r.stderr


def test_gc_pause_restores_the_collector():
    sys.path.insert(0, ROOT)
    import bench
    assert gc.isenabled()
    with bench._no_gc():
        assert not gc.isenabled()
    assert gc.isenabled()
    gc.disable()
    try:
        with bench._no_gc():
            pass
        assert not gc.isenabled()        # left as the caller had it
    finally:
        gc.enable()


def test_cpu_baseline_record():
    sys.path.insert(0, ROOT)
    import bench
    from paper_2407_21255_amd import workload as wl
    affinity = os.sched_getaffinity(0)
    rec = bench.cpu_baseline(wl.KVShape(4, 256, 8, 16, 128, wl.F16), 0.2)
    assert rec["kind"] == "oracle" and rec["cores"] == 1 and rec["unit"] == "GB/s"
    assert rec["value"] > 0 and "round trips" in rec["sample"]
    assert os.sched_getaffinity(0) == affinity        # pinning undone


def test_traffic_follows_what_the_kernels_run(tmp_path, monkeypatch):
    """The measured traffic is keyed to every source and setting that
    decides the swap launches: a changed store rule, a changed launch
    setting or a grid cap each give another key, so the bench line reports
    traffic as null until the counters are taken again."""
    import shutil
    sys.path.insert(0, ROOT)
    import bench
    csrc = os.path.join(ROOT, "paper_2407_21255_amd", "csrc")
    copy = tmp_path / "paper_2407_21255_amd" / "csrc"
    shutil.copytree(csrc, copy)
    base = bench._kernel_hash()
    assert bench._kernel_hash(str(tmp_path)) == base
    h = copy / "swap_kernels.h"
    text = h.read_text()
    assert "kNtPoolStoreMinBytes = 2ull << 30" in text
    h.write_text(text.replace("kNtPoolStoreMinBytes = 2ull << 30", "kNtPoolStoreMinBytes = 1ull << 30"))
    changed = bench._kernel_hash(str(tmp_path))
    assert changed != base
    for wl in ("llama70b_hbm", "llama8b_hbm"):
        assert bench.MEASURED_TRAFFIC.get((wl, changed)) is None
    monkeypatch.setenv("AQUA_UNIT_BYTES", "32768")
    assert bench._kernel_hash() != base
    monkeypatch.delenv("AQUA_UNIT_BYTES")
    assert bench._kernel_hash(max_workgroups=256) != base
    assert bench._kernel_hash() == base


def test_slice_options_parse_and_label_the_roofline():
    """--slice-streams and --slice-legs take only their documented values,
    and the slice roofline names what was issued and on how many streams."""
    r = _run(["--slice-streams", "3"])
    assert r.returncode == 2 and "--slice-streams" in r.stderr
    r = _run(["--slice-legs", "both_ways"])
    assert r.returncode == 2 and "--slice-legs" in r.stderr
    sys.path.insert(0, ROOT)
    import bench
    both2 = bench._slice_kernel({"slice_streams": 2, "slice_legs": "both"}, host=False)
    assert both2 == "gather and scatter of a slice, on two streams (sharing HBM)"
    assert "one link direction each" in bench._slice_kernel({}, host=True)
    assert bench._slice_kernel({"slice_streams": 1, "slice_legs": "both"}, False) == \
        "gather then scatter of a slice, on one stream"
    assert bench._slice_kernel({"slice_legs": "out"}, False) == "gather of a slice"
    assert bench._slice_kernel({"slice_legs": "in"}, True) == "scatter of a slice"
