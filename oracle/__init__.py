"""CPU oracle of ADEPT's early-exit hot path -- TEST INFRASTRUCTURE ONLY.

Only the tests, the package smoke check and the bench's CPU-baseline leg may
import this package.  It shares no code with the HIP implementation.
"""
from . import accounting, adept_oracle, brute_force  # noqa: F401
