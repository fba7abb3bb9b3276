"""Oracle for the IOS hot path — TEST INFRASTRUCTURE ONLY.

Plain, slow, independent CPU implementations of what the library computes:

* ``evaluator``: the activations of a block, by direct fp64 convolution /
  pooling loops (C, built with gcc) and numpy elementwise sums.
* ``schedule``: the IOS dynamic program (Algorithm 1), a brute-force
  enumerator of every stage partition, and the pruning / merge rules.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  It shares no code with the library and
imports nothing from it; the seeded inputs come from ``workloads``.
"""
