"""CPU oracle for the Conduit refresh step (test infrastructure only).

Only the test suite, the smoke check and the benchmark's CPU-baseline leg may
import this package; the HIP product path never does.
"""
from . import conduit_oracle  # noqa: F401
