"""The runtime option the package sets when imported (host logic, no GPU).

Streams that wait for the copy engines should be held by the command
processor, which the HIP runtime does only when GPU_STREAMOPS_CP_WAIT=1 is
in the environment before it starts.  Each case runs in a fresh interpreter,
since the package is imported once per process.
"""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

PROBE = r"""
import os, sys, warnings
sys.path.insert(0, {root!r})
import torch
if {started}:
    torch.cuda.is_initialized = lambda: True
with warnings.catch_warnings(record=True) as caught:
    warnings.simplefilter("always")
    import paper_2407_21255_amd
late = [w for w in caught if issubclass(w.category, RuntimeWarning)
        and "GPU_STREAMOPS_CP_WAIT" in str(w.message)]
print(os.environ.get("GPU_STREAMOPS_CP_WAIT"), len(late))
"""


def _probe(started: bool, env_value=None):
    env = dict(os.environ)
    env.pop("GPU_STREAMOPS_CP_WAIT", None)
    if env_value is not None:
        env["GPU_STREAMOPS_CP_WAIT"] = env_value
    out = subprocess.run(
        [sys.executable, "-c", PROBE.format(root=ROOT, started=started)],
        env=env, capture_output=True, text=True, timeout=300, check=True)
    value, warned = out.stdout.split()[-2:]
    return value, int(warned)


def test_import_before_the_runtime_starts_sets_the_option_silently():
    assert _probe(started=False) == ("1", 0)


def test_import_after_the_runtime_started_warns():
    assert _probe(started=True) == ("1", 1)


def test_a_value_from_the_environment_is_kept():
    assert _probe(started=True, env_value="0") == ("0", 0)
