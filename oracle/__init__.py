"""CPU oracle for the subspace-network codec -- test infrastructure only.

Importable by the test suite, the smoke check and the benchmark's CPU-baseline
leg; never by the product path.
"""
from . import ssn_oracle  # noqa: F401
