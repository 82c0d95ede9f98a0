"""Float64 CPU oracle of the counter-causal refresh-scoring pass.

TEST INFRASTRUCTURE ONLY: imported by the tests, the smoke check and the
benchmark's CPU-baseline leg; never by the library's product path.
"""
from .cc_oracle import *  # noqa: F401,F403
