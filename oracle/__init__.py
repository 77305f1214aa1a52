"""CPU oracle of the suffix restore.  Test infrastructure only: imported by
the test suite, the smoke check and the benchmark's CPU-baseline leg, never by
the product path."""
from .restore import *  # noqa: F401,F403
