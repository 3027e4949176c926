"""CPU oracle of the EpiKV eviction step -- test infrastructure only.

Only the tests, the smoke check and the benchmark's CPU-baseline leg may
import this package.  It shares no code with the HIP library.
"""
from .epikv_ref import *  # noqa: F401,F403
from .epikv_ref import READINGS, BUDGET_ERROR  # noqa: F401
