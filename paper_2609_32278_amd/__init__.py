"""kvx: prefix-extend attention over a paged KV pool for AMD MI355X (gfx950).

The compute path lives in ``libkvx.so`` (hand-written HIP kernels behind a C ABI,
declared in ``include/kvx.h``); ``paper_2609_32278_amd.kvx`` is its thin ctypes
binding and ``paper_2609_32278_amd.workloads`` generates seeded synthetic batches.
``agent_replay`` drives the prefix cache and the kernels through a synthetic
multi-agent workload; ``spill_model`` measures reload against recompute.
Importing the package loads nothing native; the binding loads the library on
first use and raises if it has not been built.
"""

__all__ = ["kvx", "workloads", "agent_replay", "spill_model"]
