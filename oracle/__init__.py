"""fp64 CPU oracle of the GMC boundary operator (test infrastructure only).

Only tests/, the smoke check and the benchmark's CPU-baseline leg import this
package; the HIP product path never does.
"""
from .gmc_oracle import *  # noqa: F401,F403
from .gmc_oracle import GmcParams, READINGS  # noqa: F401
