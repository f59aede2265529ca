"""fp64 CPU oracle of the batched row softmax (forward and backward), of the batched matrix
products around it, and checks of the slice schedules.

TEST INFRASTRUCTURE ONLY. Only tests/, __graft_entry__.smoke() and bench.py's cpu_baseline
leg may import this package. It shares no code with the HIP library
(paper_2002_07062_amd), and neither imports the other; inputs for both come from the
stand-alone seeded generators in workloads.py.

Pins (what checks the oracle against something other than itself) live in
tests/test_oracle.py and tests/test_plan_checks.py; every function here has at least one.
"""

from . import gemm, plan_checks
from .softmax import (DTYPE_CODE, build, softmax, softmax_backward, softmax_backward_rows,
                      softmax_rows)

__all__ = ["DTYPE_CODE", "build", "gemm", "plan_checks", "softmax", "softmax_backward",
           "softmax_backward_rows", "softmax_rows"]
