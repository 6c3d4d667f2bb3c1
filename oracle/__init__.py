"""CPU oracle for the DELTA decode-attention hot path — TEST INFRASTRUCTURE.

Imported only by the tests, the smoke check and the benchmark's CPU-baseline leg. It shares no
code with the HIP library and the library never calls it.
"""
from . import delta_oracle, accept  # noqa: F401
