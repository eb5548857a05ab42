"""CPU oracle for reachable-state weighted FST composition.

TEST INFRASTRUCTURE ONLY: imported by the test suite, the package smoke check
and the CPU-baseline leg of the benchmark, never by the product path.  It
shares no code with the HIP implementation; see ``fst_oracle.cpp`` for what it
computes and the readings it takes.
"""
from .oracle import (OracleError, OracleResult, build, compose, compose_eps, expand_pairs,
                     library_path)

__all__ = ["OracleError", "OracleResult", "build", "compose", "compose_eps", "expand_pairs",
           "library_path"]
