"""MI355X-native KV page swap: the gather (swap-out) and scatter (swap-in)
of a paged KV cache that a time-sliced, preemptive LLM scheduler issues at
every context switch (Aqua, ASPLOS '25, section 7).

Modules:
  aqua      ctypes binding of the C ABI (include/aqua.h); loads libaqua.so.
  workload  seeded synthetic inputs (pools, block tables, schedules).
  build     in-tree build of libaqua.so (hipcc, gfx950) and the host core.

Importing the package loads nothing native; ``aqua.load()`` does, and fails
loudly if the library has not been built.
"""
