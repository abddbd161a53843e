"""CPU oracle — test infrastructure, not part of the product path.

Plain, slow, obviously-correct reimplementation of what the GPU path computes:

* ``forward``  — fp64 numpy transformer forward (GPT- and LLaMA-style decoders);
* ``costs``    — analytic flops and algorithmic HBM bytes per kernel;
* ``planner``  — the tensor-granular prefetch/evict policy replayed on a trace;
* ``checker``  — semantic validation of any transfer schedule;
* ``brute``    — exhaustive search on tiny instances (least demand fetches,
  least makespan in the unit-time prefetching model) and the timing of a
  schedule in that model.

Only the tests, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  It shares no code with the HIP path and
imports nothing from it; the only common input is the seeded workload module.
"""
