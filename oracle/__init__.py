"""CPU oracle for candidate-schedule evaluation (test infrastructure only).

Only the tests, the smoke check and the benchmark's CPU-baseline leg may
import this package. It never serves the product path.
"""
from .oracle import OraclePlan, build_oracle  # noqa: F401
