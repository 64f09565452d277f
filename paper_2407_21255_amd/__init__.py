"""MI355X-native KV page swap: the gather (swap-out) and scatter (swap-in)
of a paged KV cache that a time-sliced, preemptive LLM scheduler issues at
every context switch (Aqua, ASPLOS '25, section 7).

Modules:
  aqua      ctypes binding of the C ABI (include/aqua.h); loads libaqua.so.
  workload  seeded synthetic inputs (pools, block tables, schedules).
  build     in-tree build of libaqua.so (hipcc, gfx950) and the host core.

Importing the package loads nothing native (it only sets one HIP runtime
option, below); ``aqua.load()`` does, and fails loudly if the library has
not been built.
"""
import os as _os
import sys as _sys

# The staged host path and host-side migrations make streams wait for the
# copy engines (hipStreamWaitValue64).  With this runtime setting the command
# processor holds such a stream; without it the runtime keeps a one-wave
# kernel resident for the wait, which slows kernels that fill every compute
# unit once.  It takes effect only if set before the HIP runtime starts, so
# it is set when the package is imported, unless the environment says
# otherwise.  Imported after torch has started the GPU, the setting comes too
# late: the waits stay correct, and a warning says they cost compute units.
if "GPU_STREAMOPS_CP_WAIT" not in _os.environ:
    _torch = _sys.modules.get("torch")
    if _torch is not None and _torch.cuda.is_initialized():
        import warnings as _warnings

        _warnings.warn(
            "paper_2407_21255_amd was imported after the HIP runtime started; "
            "set GPU_STREAMOPS_CP_WAIT=1 in the environment (or import this "
            "package before the first GPU call) so that stream waits on the "
            "copy engines do not keep a kernel resident",
            RuntimeWarning, stacklevel=2)
    _os.environ["GPU_STREAMOPS_CP_WAIT"] = "1"
