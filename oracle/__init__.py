"""fp64 CPU oracle of the SpeContext decode-step hot path (test infrastructure).

Only the tests, the smoke check and the benchmark's CPU-baseline leg import
this package; the product library never does.
"""
from .spec_oracle import *  # noqa: F401,F403
from .spec_oracle import __all__  # noqa: F401
