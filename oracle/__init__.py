"""CPU oracle for the multi-table embedding-bag lookup -- TEST INFRASTRUCTURE ONLY.

Plain, slow and obviously correct NumPy implementations of what the GPU path
computes, written from the paper (Ruggeri et al., "Deep Recommender Models
Inference: Automatic Asymmetric Data Flow Optimization"):

* ``pool``  -- the pooled lookup itself (Sec. II-B definition, sum reduction as in
  Sec. IV-A), accumulated in float64 and rounded once to float32.
* ``index`` -- the index transforms the strategies apply (chunk offset subtraction
  of Sec. III-B, hot-row membership, tile deduplication, range checking).
* ``plan``  -- the planner: the linear cost model of Eq. (2) extended to the four
  GPU strategies and the greedy asymmetric mapping of Sec. III-B (steps 1-4),
  followed literally so that two independent implementations can be compared
  byte for byte.  Parity unpinned against the paper (it prints no worked plan);
  pinned by invariants, special cases and scheduling bounds in the tests.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The library under
``paper_2507_01676_amd`` never imports it and shares no code with it.
"""
from . import index, plan, pool  # noqa: F401
