"""CPU oracle of EDiT's outer synchronization step -- TEST INFRASTRUCTURE.

Only the tests, the smoke check and the benchmark's CPU-baseline leg may
import this package.  The product library never does; it shares no code
with it.  See oracle/edit_oracle.c for the statement of the step.
"""
from .oracle import (  # noqa: F401
    AE, GC, WA, OracleConfig, OracleUnit, bf16_bits_to_f32, f32_to_bf16_bits, library_path,
)
