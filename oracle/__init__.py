"""CPU oracle for the LayUp layer-wise backward -> update -> gossip-mix step.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path imports this package:
only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may use it.  It shares no code with the HIP library.

The oracle is plain numpy in float64.  Where the GPU path stores a tensor in
bfloat16 the oracle rounds to bfloat16 (round-to-nearest-even) at the same
point; where the GPU path keeps float32 the oracle keeps float64, except for
the optimizer outputs (parameters, momentum, second moment), which are the
float32 master state of the method and are rounded to float32.
"""
from .layup_ref import *  # noqa: F401,F403
