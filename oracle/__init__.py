"""Test infrastructure: the fp64 CPU oracle of the MALT / MALTER step.

Only the tests, the package smoke check and the benchmark's CPU-baseline leg
may import this package.  It shares no code with the HIP library.
"""
from .malt_oracle import (  # noqa: F401
    NS_A, NS_B, NS_C, NS_EPS, NS_STEPS, VARIANT_MALT, VARIANT_MALTER,
    OracleHparams, OracleState, StepIntermediates, newton_schulz, oracle_init,
    oracle_step, polar_svd, rel_fro,
)
