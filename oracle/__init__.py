"""fp64 CPU oracle for the micro-batch pipeline stage with checkpointing.

TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT.  Only the tests, the smoke
check and the benchmark's CPU-baseline leg may import or call anything in
this package; the HIP path never does, and shares no code with it.  The one
module both sides use is `workloads` (network structure and seeded inputs),
which holds none of the method's arithmetic.

  ops       float64 definitions of every layer operation and its adjoint
  network   full-batch forward/backward of a layer sequence (the definition
            the pipeline must reproduce), with an optional bf16-storage mode
  pipeline  the paper's micro-batch / clock-cycle / checkpoint decomposition,
            used to pin the invariants of Sec. 2 and Sec. 2.1
  params    seeded parameters of a network as float64 arrays

Parity status: every function here is pinned by tests/test_oracle_*.py
(closed forms, adjoint identities, finite differences, torch-CPU float64
cross-checks, micro-batch and recompute invariants).  Nothing is unpinned.
"""
from . import ops, network, pipeline  # noqa: F401
from .params import net_params  # noqa: F401
