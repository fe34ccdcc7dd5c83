"""CPU oracle for row-centric CNN training (LR-CNN, arXiv 2401.11471).

TEST INFRASTRUCTURE, not part of the product. Only ``tests/``,
``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of ``bench.py`` may
import it. It shares no code with the HIP library (``paper_2401_11471_amd``)
and neither side imports the other; both take their seeded inputs from
``workloads``.

Modules:
  column  -- float64 layer-by-layer training (the definition the method must
             reproduce), with optional bfloat16 storage emulation
  bf16    -- round-to-nearest-even to bfloat16 from the format's definition
  rows    -- the row-partitioned runner (two-phase sharing and overlapping
             partitioning) with its own interval arithmetic
  brute   -- scalar loops for tiny shapes that pin ``column``
  head    -- classifier head, softmax cross-entropy and SGD of a full training
             step (Algorithm 1's fully connected FP/BP, loss and update)

Parity status: every function is pinned by tests in ``tests/test_oracle_*``
(brute force, library routines, adjoint identities, finite differences,
partition invariance, the paper's worked shape examples). The bf16 emulation
mode's rounding points are a reading of the paper (it states no precision);
the rounding routine itself is pinned against a library conversion.
"""
