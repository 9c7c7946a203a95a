"""CPU oracle for the large-batch actor-critic update (TEST INFRASTRUCTURE ONLY).

A plain, slow, float64 NumPy implementation of one update step of the method's
network-update process (Section 3.2: a single large-batch updater that trains
the actor and the twin critics with their target networks; SAC is the worked
example, TD3 the alternative of Section 4.2.4, Fig. 8). The paper prints no update
equations, so each step follows the published SAC (Haarnoja et al., 2018) and
TD3 (Fujimoto et al., 2018) algorithms; the readings taken where the paper is
silent are listed in the module docstrings.

Only the test-suite, the package's smoke check and the benchmark's CPU-baseline
leg may import this package. It shares no code with the HIP implementation and
never imports it.

Modules
  philox  counter-based Philox4x32-10 streams, replay indices, normal deviates, init
  bf16    round-to-nearest-even to bfloat16 (operand emulation for bf16 workloads)
  nets    MLP parameter layout, forward and backward
  update  the Oracle class: replay ring, SAC / TD3 step, Adam, Polyak, loss records
"""
from .update import Oracle  # noqa: F401
