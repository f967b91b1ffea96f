"""fp64 CPU oracle of the block-sparse attention path (test infrastructure only).

Imported by the tests, the smoke check and the benchmark's CPU-baseline leg;
never by the library.
"""
from .spade_oracle import *  # noqa: F401,F403
