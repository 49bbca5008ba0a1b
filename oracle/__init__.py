"""CPU oracle for the Compass hot path — TEST INFRASTRUCTURE ONLY.

Only the test-suite, the package smoke check and the benchmark's CPU-baseline
leg may import this package. It shares no code with the HIP path.
"""
from .compass_oracle import *  # noqa: F401,F403
