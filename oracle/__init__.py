"""Float64 CPU oracle for the MAPL boundary codec and the SPEL Stiefel step.

TEST INFRASTRUCTURE ONLY.  Nothing in the product package imports, links or
executes anything under this directory.  The only callers are ``tests/``,
``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of ``bench.py``.

The oracle is written from the paper (Manifold Aware Projection Learning,
Sec. 3.2 Eqs. 1-3, Sec. 3.3 Eqs. 4-7 and Algorithm 1, Sec. 3.5) as plain,
slow, obviously-correct NumPy in float64.  It shares no code, headers, tables
or constant generators with the HIP path; only the seeded input generator
(``paper_2606_05484_amd.synth``, which holds none of the method's arithmetic)
feeds both sides.

Modules
  precision      bf16 / fp32 rounding used to mirror operand precision
  codec          Eq. 1 (encode), Eq. 2 (decode), RVQ (Sec. 3.5), backward
  polar_schedule greedy minimax odd-quintic schedule (PolarExpress, Sec. 3.3)
  spel           Eqs. 4-7: tangent projection, momentum, LMO, retraction
"""

