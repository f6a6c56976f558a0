"""CPU oracle for the fixed-cost drafting step (test infrastructure only).

A plain, slow, fp64 numpy statement of what the drafting step computes:

* ``oracle.views``  -- the fixed-size context views (Sec. 2.2, Eq. 5 and the
  incremental merge of App. A.2, Eq. 10-11): recent K/V window, global
  summary (M, eta) and the boundary hidden states.
* ``oracle.draft``  -- the block-diffusion drafter forward (Sec. 2.3, Eq. 4,
  Eq. 6, App. A.1, App. B.1) producing the base logits z^(0).
* ``oracle.sample`` -- per-position sampling of the factorised proposal
  (Eq. 8) by Gumbel-max over seeded counter-based noise.

Only the tests, the smoke check and the benchmark's CPU-baseline leg may
import this package. The GPU library never calls it and shares no code with
it; the two meet only through the seeded inputs of ``synth``.

Every function here is pinned by ``tests/test_oracle_*.py`` against something
other than itself (closed forms, brute force, library routines, invariants).
"""
