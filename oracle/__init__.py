"""CPU oracle of the PrHS decode hot path (test infrastructure only).

Only the test suite, the package smoke check and the benchmark's CPU-baseline
leg may import this package.  It shares no code with the HIP library.
"""

from .prhs_oracle import *  # noqa: F401,F403
from .prhs_oracle import brute_force_topk_mass  # noqa: F401
