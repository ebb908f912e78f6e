"""CPU oracle for the tuning hot path (test infrastructure only).

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  It shares no code with the HIP library
(``paper_2406_20037_amd``) and neither imports the other; the only common
module is ``synthdata`` (seeded inputs, no method arithmetic).

Contents:

* ``kernels``  -- fp64 direct conv2d and matmul (plain C, ``oracle_kernels.c``).
* ``space``    -- the schedule lattice of each kernel family: value lists,
  clipping, validity, launch geometry, mixed-radix key, neighbourhood.
* ``sampler``  -- the seeded exploration sampler (own SplitMix64).
* ``droplet``  -- Droplet Search coordinate descent and the combined
  explore-then-exploit procedure, plus the rank-sum convergence test.
* ``exploiters`` -- the strategies Droplet Search is compared with as the
  exploitation phase (Random, Grid, GA; Section 3, RQ4).
* ``task_scheduler`` -- one trial budget split across the layers of a network
  (Section 2.1, Termination in Ansor), then Droplet Search per layer.

Parity status of each part is stated in its module header.
"""
