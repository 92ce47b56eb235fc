"""CPU oracle of the RW-TTT fast-weight READ/WRITE path (test infrastructure).

Only the test suite, the smoke check and the benchmark's CPU-baseline leg may
import this package.  The product library never does, and shares no code with
it; both sides only share the seeded input generators in ``rwttt_inputs``.
"""

from .rwttt_oracle import *  # noqa: F401,F403
