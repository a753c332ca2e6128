"""CPU oracle of the Mira MoE expert step: test infrastructure, not product code.

Only the tests, the smoke check and the benchmark's CPU-baseline leg import
this package.  It shares no code with the GPU library.
"""
from .mira_oracle import *  # noqa: F401,F403
from .mira_oracle import __all__  # noqa: F401
