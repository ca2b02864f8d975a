"""CPU oracle for the tied-trit-plane expert dot pass. TEST INFRASTRUCTURE ONLY:
imported by tests, the smoke check and the benchmark's CPU-baseline leg, never by the
product path (the HIP library and its binding)."""
from .oracle import Oracle, OracleError, expert_getter, get  # noqa: F401
